// hb_gemm.hip -- the GEMM strategy (Algorithm 1 with the tensors of Table 3,
// Sec. 4.1) on the int8 matrix cores of gfx950.
//
// Algorithm 1 multiplies X by A (a selection of one feature per decision
// node), compares with B, multiplies the 0/1 outcome by C (+1 for leaves in
// a node's left subtree, -1 in its right subtree), tests equality with D and
// maps the one-hot leaf through E. Here:
//   * X.A < B is evaluated as a gather and a compare (never a float product,
//     which would turn a NaN or infinite feature into NaN for every node);
//     the outcome is encoded as the int8 value 64 (true) or 0;
//   * the path product runs as v_mfma_i32_16x16x64_i8 with the A operand
//     4*C^T (leaves x decision nodes) and the B operand the encoded outcomes
//     (decision nodes x rows), so every product term is 0 or +-256;
//   * the accumulator starts at bias[l] = l - 256*D[l], so it ends at
//     256*((T.C)_l - D_l) + l. (T.C)_l <= D_l with equality only for the
//     selected leaf, hence the selected leaf's column is the unique
//     non-negative value, and the maximum over columns is that column index:
//     the "== D" test and the leaf lookup of the one-hot product collapse
//     into one v_max per accumulator element;
//   * the leaf's value and caller id are then gathered (E of Table 3).
// Lane layout of v_mfma_i32_16x16x64_i8 (checked on the device): lane l
// supplies A[m = l%16][k = 16(l/16) .. +15] and B[k = 16(l/16) .. +15][n = l%16]
// and receives D[4(l/16) + i][n = l%16], i = 0..3.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <string>

#include "hb_device.h"

namespace hb {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Rows per workgroup: 64 per wave, 8 waves (two per SIMD, so one wave's
// predicate phase overlaps another's matrix phase) when LDS allows, else 4.
// The feature tile's stride is the row count + 8 (spreads lane groups over banks).
constexpr int kCtPad = 16;                 // bytes appended to each C^T row in LDS
constexpr int kTG = 4;                     // trees per staged chunk of node records
constexpr int kIdGroup = 32;               // trees per leaf-id flush

struct GemmArgs {
  const float *X;
  int64_t n_rows;
  int32_t F;                // feature-tile columns
  int32_t Fs;               // row stride of X (input columns)
  const int32_t *cols;      // tile column -> input column, or nullptr
  int32_t *leaf_ids;
  OutArgs out;
  const int32_t *tree_class;
  int32_t LD;
  const uint2 *node;        // [T][k_pad] {threshold bits, feature}
  const int32_t *shape;     // [T]
  const int8_t *ct;         // [S][l_pad][k_pad]
  const int32_t *bias;      // [S][l_pad]
  const float *leaf_value;  // [T][l_pad][LD]
  const int32_t *leaf_id;   // [T][l_pad]
  int32_t k_pad, l_pad;
  int32_t ids_vec;
  // tree split (small batches, the 16-row tile kernels): workgroup (x, y) takes
  // trees [y * split, min((y + 1) * split, T)) of row tile x and stores its
  // raw sums in partial[y][row][K]; 0 = every tree, rows finished in place
  int32_t split;
  double *partial;
};

// LDS bytes of one tree's node records: groups of 16 records (128 B) are
// followed by 16 B of padding, so the four lane groups of a wave, which read
// 16 consecutive records each, start 36 banks apart.
__host__ __device__ constexpr int node_lds_bytes(int k_pad) { return k_pad * 9; }
__host__ __device__ constexpr int node_lds_off(int k) { return k * 8 + (k / 16) * 16; }

__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ int hmax4(v4i v) { return max(max(v[0], v[1]), max(v[2], v[3])); }

// Node records of one chunk of kTG trees, held in registers between their
// global load (issued before the current chunk is walked) and their store to
// LDS (after it), in the padded layout; 16 B (two records) per lane per step.
// Native vectors so they stay in VGPRs.
template <int ROWS>
struct NodePrefetch {
  static constexpr int PER = kTG * 256 / 2 / ROWS;  // k_pad <= 256
  u32x4 v[PER];
  __device__ __forceinline__ void load(const GemmArgs &a, int t0) {
    const int per_tree16 = a.k_pad / 2;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = min(i * ROWS + (int)threadIdx.x, kTG * per_tree16 - 1);
      const int g = u / per_tree16;
      const int q = u - g * per_tree16;
      const int t = min(t0 + g, a.out.T - 1);
      v[i] = reinterpret_cast<const u32x4 *>(a.node + (size_t)t * a.k_pad)[q];
    }
  }
  __device__ __forceinline__ void store(const GemmArgs &a, unsigned char *dst) const {
    const int per_tree16 = a.k_pad / 2;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = i * ROWS + (int)threadIdx.x;
      if (u < kTG * per_tree16) {
        const int g = u / per_tree16;
        const int q = u - g * per_tree16;
        *reinterpret_cast<u32x4 *>(dst + g * node_lds_bytes(a.k_pad) + node_lds_off(2 * q)) = v[i];
      }
    }
  }
};

// KB: 64-node slices of the decision-node dimension; KMODE: 0 scalar leaves
// and one output, 1 scalar leaves with a class per tree, 2 vector leaves.
template <int KB, bool CT_LDS, bool X_LDS, int KMODE, int ROWS, bool COLS = false>
__global__ __launch_bounds__(ROWS) void gemm_kernel(GemmArgs a) {
  constexpr int KMAX = KMODE == 0 ? 1 : HB_MAX_OUTPUTS;
  constexpr int XS = ROWS + 8;
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ __align__(16) int4 idstage[ROWS / 64][16 * (kIdGroup / 4)];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int g4 = lane >> 4;  // lane group: k slice of the operands, leaf quad of the result
  const int r16 = lane & 15;
  const int wave = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * ROWS;
  const int64_t r0w = r0 + wave * 64;
  const int64_t row = r0w + lane;  // the row this lane owns after the reduction
  const bool valid = row < a.n_rows;
  const int LT = a.l_pad / 16;
  const int ct_stride = a.k_pad + kCtPad;

  // ---- LDS carve-up: [feature tile][C^T][bias][node chunks x2]
  size_t off = 0;
  float *xs = reinterpret_cast<float *>(smem);
  if (X_LDS) off += ((size_t)a.F * XS * 4 + 15) / 16 * 16;
  int8_t *cts = reinterpret_cast<int8_t *>(smem + off);
  int32_t *bias_s = nullptr;
  if (CT_LDS) {
    off += (size_t)a.l_pad * ct_stride;
    bias_s = reinterpret_cast<int32_t *>(smem + off);
    off += (size_t)a.l_pad * 4;
  }
  unsigned char *nodes = smem + off;
  const int chunk_bytes = kTG * node_lds_bytes(a.k_pad);

  if (X_LDS) {
    for (int f = 0; f < a.F; ++f)
      xs[f * XS + tid] = (r0 + tid < a.n_rows) ? xval(a.X + (r0 + tid) * a.Fs, a.cols, f) : 0.0f;
  }
  if (CT_LDS) {
    const int row16 = a.k_pad / 16;
    for (int u = tid; u < a.l_pad * row16; u += ROWS) {
      const int l = u / row16;
      const int q = u - l * row16;
      *reinterpret_cast<u32x4 *>(cts + (size_t)l * ct_stride + q * 16) =
          reinterpret_cast<const u32x4 *>(a.ct + (size_t)l * a.k_pad)[q];
    }
    for (int u = tid; u < a.l_pad; u += ROWS) bias_s[u] = a.bias[u];
  }
  {
    NodePrefetch<ROWS> first;
    first.load(a, 0);
    first.store(a, nodes);
  }
  lds_sync();

  double acc[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) acc[k] = 0.0;
  int32_t ids[kIdGroup];
#pragma unroll
  for (int q = 0; q < kIdGroup; ++q) ids[q] = 0;

  const float *xrow[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    const int64_t rr = r0w + rt * 16 + r16;
    xrow[rt] = a.X + (rr < a.n_rows ? rr : a.n_rows - 1) * a.Fs;
  }

  const int n_chunks = (a.out.T + kTG - 1) / kTG;
  for (int c = 0; c < n_chunks; ++c) {
    const unsigned char *cur = nodes + (c & 1) * chunk_bytes;
    const bool more = c + 1 < n_chunks;
    NodePrefetch<ROWS> next;
    next.load(a, more ? (c + 1) * kTG : c * kTG);
    __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the walk
    for (int tg = 0; tg < kTG; ++tg) {
      const int t = c * kTG + tg;
      if (t >= a.out.T) break;  // uniform
      const unsigned char *nb = cur + tg * node_lds_bytes(a.k_pad);
      // ---- B operand: encoded outcomes of this lane's 16 nodes per slice, 4 row tiles
      v4i bop[4][KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const unsigned char *rb = nb + node_lds_off(kb * 64 + 16 * g4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {  // four records -> one byte-packed dword per row tile
          const u32x4 v0 = *reinterpret_cast<const u32x4 *>(rb + q * 32);
          const u32x4 v1 = *reinterpret_cast<const u32x4 *>(rb + q * 32 + 16);
          const uint2 rec[4] = {make_uint2(v0[0], v0[1]), make_uint2(v0[2], v0[3]), make_uint2(v1[0], v1[1]),
                                make_uint2(v1[2], v1[3])};
#pragma unroll
          for (int rt = 0; rt < 4; ++rt) {
            uint32_t w = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              const float x = X_LDS ? xs[rec[b].y * XS + wave * 64 + rt * 16 + r16] : xget<COLS>(xrow[rt], a.cols, rec[b].y);
              w |= (x < as_float(rec[b].x) ? 0x40u : 0u) << (8 * b);
            }
            bop[rt][kb][q] = (int)w;
          }
        }
      }
      // ---- path product and "== D": running maximum of 256 (T.C - D) + l
      const int s = CT_LDS ? 0 : a.shape[t];
      const int8_t *ctg = a.ct + (size_t)s * a.l_pad * a.k_pad;
      const int32_t *bg = a.bias + (size_t)s * a.l_pad;
      int best[4] = {INT_MIN, INT_MIN, INT_MIN, INT_MIN};
      for (int lt = 0; lt < LT; ++lt) {
        v4i b4;
        if (CT_LDS)
          b4 = *reinterpret_cast<const v4i *>(bias_s + lt * 16 + 4 * g4);
        else
          b4 = *reinterpret_cast<const v4i *>(bg + lt * 16 + 4 * g4);
        v4i d[4] = {b4, b4, b4, b4};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          v4i av;
          if (CT_LDS)
            av = *reinterpret_cast<const v4i *>(cts + (size_t)(lt * 16 + r16) * ct_stride + kb * 64 + 16 * g4);
          else
            av = *reinterpret_cast<const v4i *>(ctg + (size_t)(lt * 16 + r16) * a.k_pad + kb * 64 + 16 * g4);
#pragma unroll
          for (int rt = 0; rt < 4; ++rt) d[rt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bop[rt][kb], d[rt], 0, 0, 0);
        }
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) best[rt] = max(best[rt], hmax4(d[rt]));
      }
      // rows are spread over the four lane groups: combine them
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        best[rt] = max(best[rt], __shfl_xor(best[rt], 16));
        best[rt] = max(best[rt], __shfl_xor(best[rt], 32));
      }
      // lane l owns row l of the wave (row tile l/16, row l%16)
      int col = g4 == 0 ? best[0] : g4 == 1 ? best[1] : g4 == 2 ? best[2] : best[3];
      col = min(max(col, 0), a.l_pad - 1);  // a valid tree always yields a column in range
      const size_t lrec = (size_t)t * a.l_pad + (size_t)col;
      if (KMODE == 2) {
#pragma unroll
        for (int k = 0; k < KMAX; ++k)
          if (k < a.LD) acc[k] += (double)a.leaf_value[lrec * a.LD + k];
      } else if (KMODE == 0) {
        acc[0] += (double)a.leaf_value[lrec];
      } else {
        const int cls = __builtin_amdgcn_readfirstlane(a.tree_class[t]);
        const double v = (double)a.leaf_value[lrec];
#pragma unroll
        for (int k = 0; k < KMAX; ++k)
          if (k == cls) acc[k] += v;
      }
      const int slot = t % kIdGroup;
#pragma unroll
      for (int q = 0; q < kIdGroup; ++q)
        if (q == slot) ids[q] = a.leaf_id[lrec];
      if (a.leaf_ids && (slot == kIdGroup - 1 || t == a.out.T - 1))
        flush_ids<kIdGroup>(a.leaf_ids, a.n_rows, a.out.T, a.ids_vec, false, idstage[wave], ids, r0w, t - slot);
    }
    // the other buffer held chunk c - 1, which every wave finished before the
    // barrier that ended it
    if (more) next.store(a, nodes + ((c + 1) & 1) * chunk_bytes);
    lds_sync();
  }
  if (valid) finish_row<KMAX>(a.out, acc, row);
}

// ---------------------------------------------------------------------------
// Software-pipelined variant for trees with 193..255 decision nodes and
// 241..256 leaves (perfect depth-8 trees): KB = 4 slices, 16 leaf tiles.
// While the 16 matrix instructions of leaf tile lt of tree t run, the wave
// builds slice lt of tree t+1's predicate operand (one 64-node slice and four
// records per lane group per tile), so the matrix cores and the vector ALUs
// work at the same time within one wave. Node records are read from the L1/L2
// copy of the tables two slices ahead (four records per lane group, one
// 128-byte line per group), so no staging and no barrier is needed in the loop.

struct PipeRecs {
  u32x4 lo, hi;  // four node records {threshold bits, feature}
};

__device__ __forceinline__ PipeRecs pipe_load(const GemmArgs &a, int t, int unit, int g4) {
  const int k = (unit >> 2) * 64 + 16 * g4 + 4 * (unit & 3);
  const u32x4 *p = reinterpret_cast<const u32x4 *>(a.node + (size_t)t * a.k_pad + k);
  return PipeRecs{p[0], p[1]};
}

// Encoded outcomes (bytes 0/64) of four decision nodes for the four row tiles.
template <int XS>
__device__ __forceinline__ void pipe_pred(const PipeRecs &r, const float *xs, int xrow0, v4i (&dst)[4], int q) {
  const uint32_t thr[4] = {r.lo[0], r.lo[2], r.hi[0], r.hi[2]};
  const uint32_t fea[4] = {r.lo[1], r.lo[3], r.hi[1], r.hi[3]};
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    uint32_t w = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const float x = xs[fea[b] * XS + xrow0 + rt * 16];
      w |= (x < as_float(thr[b]) ? 0x40u : 0u) << (8 * b);
    }
    dst[rt][q] = (int)w;
  }
}

template <int KMODE, int ROWS>
struct PipeState {
  static constexpr int KMAX = KMODE == 0 ? 1 : HB_MAX_OUTPUTS;
  double acc[KMAX];
};

// One tree: the path product of tree t from `cur`, and tree t+1's operand into `nxt`.
template <int KMODE, int ROWS>
__device__ __forceinline__ void pipe_tree(const GemmArgs &a, int t, const v4i (&cur)[4][4], v4i (&nxt)[4][4],
                                          const float *xs, const int8_t *cts, const int32_t *bias_s, int ct_stride,
                                          int wave, int g4, int r16, int64_t r0w, int4 *stage,
                                          PipeState<KMODE, ROWS> &st) {
  constexpr int XS = ROWS + 8;
  const int tn = min(t + 1, a.out.T - 1);
  const int xrow0 = wave * 64 + r16;
  PipeRecs r0 = pipe_load(a, tn, 0, g4);
  PipeRecs r1 = pipe_load(a, tn, 1, g4);
  int best[4] = {INT_MIN, INT_MIN, INT_MIN, INT_MIN};
#pragma unroll
  for (int lt = 0; lt < 16; ++lt) {
    const v4i b4 = *reinterpret_cast<const v4i *>(bias_s + lt * 16 + 4 * g4);
    v4i d[4] = {b4, b4, b4, b4};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const v4i av = *reinterpret_cast<const v4i *>(cts + (lt * 16 + r16) * ct_stride + kb * 64 + 16 * g4);
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) d[rt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, cur[rt][kb], d[rt], 0, 0, 0);
    }
    // slice lt of the next tree: kb = lt / 4, records 4 (lt % 4) .. +3 of each lane group
    PipeRecs r2 = r1;
    if (lt + 2 < 16) r2 = pipe_load(a, tn, lt + 2, g4);
    {
      v4i slice[4];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) slice[rt] = nxt[rt][lt >> 2];
      pipe_pred<XS>(r0, xs, xrow0, slice, lt & 3);
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) nxt[rt][lt >> 2] = slice[rt];
    }
    r0 = r1;
    r1 = r2;
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) best[rt] = max(best[rt], hmax4(d[rt]));
    // one leaf tile per scheduling region: keeps live ranges (and registers) bounded
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    best[rt] = max(best[rt], __shfl_xor(best[rt], 16));
    best[rt] = max(best[rt], __shfl_xor(best[rt], 32));
  }
  int col = g4 == 0 ? best[0] : g4 == 1 ? best[1] : g4 == 2 ? best[2] : best[3];
  col = min(max(col, 0), a.l_pad - 1);  // a valid tree always yields a column in range
  const size_t lrec = (size_t)t * a.l_pad + (size_t)col;
  if (KMODE == 2) {
#pragma unroll
    for (int k = 0; k < PipeState<KMODE, ROWS>::KMAX; ++k)
      if (k < a.LD) st.acc[k] += (double)a.leaf_value[lrec * a.LD + k];
  } else if (KMODE == 0) {
    st.acc[0] += (double)a.leaf_value[lrec];
  } else {
    const int cls = __builtin_amdgcn_readfirstlane(a.tree_class[t]);
    const double v = (double)a.leaf_value[lrec];
#pragma unroll
    for (int k = 0; k < PipeState<KMODE, ROWS>::KMAX; ++k)
      if (k == cls) st.acc[k] += v;
  }
  // leaf ids go straight out (this kernel is bound by the matrix cores, and
  // holding 32 ids per lane would cost the registers the pipeline needs)
  const int64_t row = r0w + (threadIdx.x & 63);
  if (a.leaf_ids && row < a.n_rows) a.leaf_ids[row * a.out.T + t] = a.leaf_id[lrec];
  (void)stage;
}

template <int KMODE, int ROWS>
__global__ __launch_bounds__(ROWS) void gemm_pipe_kernel(GemmArgs a) {
  constexpr int XS = ROWS + 8;
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ __align__(16) int4 idstage[ROWS / 64][16 * (kIdGroup / 4)];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int g4 = lane >> 4;
  const int r16 = lane & 15;
  const int wave = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * ROWS;
  const int64_t r0w = r0 + wave * 64;
  const int64_t row = r0w + lane;
  const int ct_stride = a.k_pad + kCtPad;
  float *xs = reinterpret_cast<float *>(smem);
  const size_t xbytes = ((size_t)a.F * XS * 4 + 15) / 16 * 16;
  int8_t *cts = reinterpret_cast<int8_t *>(smem + xbytes);
  int32_t *bias_s = reinterpret_cast<int32_t *>(smem + xbytes + (size_t)a.l_pad * ct_stride);
  for (int f = 0; f < a.F; ++f)
    xs[f * XS + tid] = (r0 + tid < a.n_rows) ? xval(a.X + (r0 + tid) * a.Fs, a.cols, f) : 0.0f;
  {
    const int row16 = a.k_pad / 16;
    for (int u = tid; u < a.l_pad * row16; u += ROWS) {
      const int l = u / row16;
      const int q = u - l * row16;
      *reinterpret_cast<u32x4 *>(cts + (size_t)l * ct_stride + q * 16) =
          reinterpret_cast<const u32x4 *>(a.ct + (size_t)l * a.k_pad)[q];
    }
    for (int u = tid; u < a.l_pad; u += ROWS) bias_s[u] = a.bias[u];
  }
  lds_sync();

  PipeState<KMODE, ROWS> st;
#pragma unroll
  for (int k = 0; k < PipeState<KMODE, ROWS>::KMAX; ++k) st.acc[k] = 0.0;
  // operand of tree 0
  v4i opa[4][4], opb[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) opa[i][j] = opb[i][j] = v4i{0, 0, 0, 0};
  const int xrow0 = wave * 64 + r16;
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    v4i slice[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) slice[rt] = opa[rt][u >> 2];
    pipe_pred<XS>(pipe_load(a, 0, u, g4), xs, xrow0, slice, u & 3);
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) opa[rt][u >> 2] = slice[rt];
  }
  for (int t = 0; t < a.out.T; ++t) {
    pipe_tree<KMODE, ROWS>(a, t, opa, opb, xs, cts, bias_s, ct_stride, wave, g4, r16, r0w, idstage[wave], st);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) opa[i][j] = opb[i][j];
  }
  if (row < a.n_rows) finish_row<PipeState<KMODE, ROWS>::KMAX>(a.out, st.acc, row);
}

// ---------------------------------------------------------------------------
// Wide rows: when 256 rows of features do not fit in LDS next to C^T (a few
// thousand input columns), a workgroup takes 16 rows, the N dimension of one
// v_mfma_i32_16x16x64_i8, and keeps C^T in registers instead of LDS: wave w
// holds the A operands of leaves 64w .. 64w + 63 (4 leaf tiles x 4 slices,
// 64 VGPRs). Per tree the four waves build the shared predicate operand
// (256 decision nodes x 16 rows, bytes 0/64) together, one 16-node block of
// one row per thread, into a double-buffered LDS tile; each wave then runs
// its 16 matrix instructions and reduces its leaves to four maxima per row
// (one per lane group), and the sixteen maxima meet in LDS. Trees go in
// pairs, one barrier per pair. Node records pass through LDS one pair ahead
// (loaded two pairs ahead); the leaf of tree t is looked up by wave t mod 4,
// whose loads are consumed when that wave's turn comes again, and the four
// waves' partial sums are added in wave order at the end. This four-wave
// kernel runs where the tile leaves room for two workgroups per CU; where it
// leaves room for one (a 16-row tile of 2,000 features), gemm_tile2_kernel
// puts eight waves on the one tile.
constexpr int kTileRows = 16;
constexpr int kTileBStride = 256 + 16;  // bytes per row of the predicate tile (spreads the 16 rows over banks)

// Row stride of the feature tile in floats: a multiple of 4 whose quotient by
// 4 is odd, so the 16 rows of one feature fall in 16 different banks.
__host__ __device__ inline int gemm_tile_xs(int F) {
  const int xs = (F + 3) & ~3;
  return (xs & 7) ? xs : xs + 4;
}

// KM: outputs a row's sums hold (1 for one output; the class count or leaf
// width rounded up to a compiled size, else HB_MAX_OUTPUTS)
template <int KMODE, int KM = (KMODE == 0 ? 1 : HB_MAX_OUTPUTS)>
struct TileLeaf {
  static constexpr int KMAX = KM;
  int t = -1;  // tree of the pending lookup, -1 none
  int cls = 0;
  int32_t id = 0;
  float v[KMODE == 2 ? KMAX : 1];
};

template <int KMODE, int KM>
__device__ __forceinline__ void tile_leaf_issue(const GemmArgs &a, TileLeaf<KMODE, KM> &p, int t, int col) {
  const size_t lrec = (size_t)t * a.l_pad + (size_t)col;
  p.t = t;
  p.id = a.leaf_id[lrec];
  if (KMODE == 2) {
#pragma unroll
    for (int k = 0; k < KM; ++k) p.v[k] = k < a.LD ? a.leaf_value[lrec * a.LD + k] : 0.0f;
  } else {
    p.v[0] = a.leaf_value[lrec];
    if (KMODE == 1) p.cls = a.tree_class[t];
  }
}

template <int KMODE, int KM>
__device__ __forceinline__ void tile_leaf_consume(const GemmArgs &a, TileLeaf<KMODE, KM> &p, double (&acc)[KM],
                                                  int64_t row) {
  if (p.t < 0) return;
  if (KMODE == 2) {
#pragma unroll
    for (int k = 0; k < KM; ++k) acc[k] += (double)p.v[k];
  } else if (KMODE == 0) {
    acc[0] += (double)p.v[0];
  } else {
#pragma unroll
    for (int k = 0; k < KM; ++k)
      if (k == p.cls) acc[k] += (double)p.v[0];
  }
  if (a.leaf_ids && row < a.n_rows) a.leaf_ids[row * a.out.T + p.t] = p.id;
  p.t = -1;
}

// Predicate operand of one tree: thread (row tid % 16, nodes 16 (tid / 16)
// .. + 15) compares its row's features with its 16 records and writes the 16
// outcome bytes (64 where x < threshold) to the tile.
__device__ __forceinline__ void tile_build1(const float *xs, int XS, const uint2 *rtab, unsigned char *bt, int tid) {
  // tid: the thread's index among the 256 that build this tree
  const int r = tid & 15, nb = tid >> 4;
  const uint2 *rec = rtab + nb * 16;
  u32x4 w;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t word = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const uint2 nr = rec[q * 4 + b];
      word |= (xs[r * XS + (int)nr.y] < as_float(nr.x) ? 0x40u : 0u) << (8 * b);
    }
    w[q] = word;
  }
  *reinterpret_cast<u32x4 *>(bt + r * kTileBStride + nb * 16) = w;
}

// The path product of one tree for this wave's 64 leaves (4 leaf tiles),
// accumulators started at the biases.
__device__ __forceinline__ void tile_product(const unsigned char *bt, const v4i (&ctr)[4][4], const v4i (&b4)[4],
                                             v4i (&d)[4]) {
  const int lane = threadIdx.x & 63, g4 = lane >> 4, r16 = lane & 15;
  v4i bop[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) bop[kb] = *reinterpret_cast<const v4i *>(bt + r16 * kTileBStride + kb * 64 + 16 * g4);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    d[j] = b4[j];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) d[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ctr[j][kb], bop[kb], d[j], 0, 0, 0);
  }
}

__device__ __forceinline__ int tile_best(const v4i (&d)[4]) {
  return max(max(hmax4(d[0]), hmax4(d[1])), max(hmax4(d[2]), hmax4(d[3])));
}

// Trees t and t+1 (t even); P = (t / 2) & 1 selects the buffers and the
// record registers. Records of trees t+4, t+5 (loaded two pairs ago) go to
// LDS for the build one pair ahead, and trees t+8, t+9 are loaded. Past the
// last tree the products and builds run on the last tree's records (clamped
// loads) and are discarded, so the pair is one straight block: the builds
// are issued while the matrix instructions execute, and only then are the
// accumulators read.
template <int KMODE, int P>
__device__ __forceinline__ void tile_pair(const GemmArgs &a, int t, const float *xs, int XS,
                                          unsigned char (*bt)[2][kTileRows * kTileBStride], uint2 (*rtab)[2][256],
                                          int (*red)[2][16][kTileRows], uint2 (&rset)[2][2], const v4i (&ctr)[4][4],
                                          const v4i (&b4)[4], TileLeaf<KMODE> &pend,
                                          double (&acc)[TileLeaf<KMODE>::KMAX], int64_t r0, int T) {
  // T: one past this workgroup's last tree
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, r16 = lane & 15;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    rtab[P][u][tid] = rset[P][u];
    rset[P][u] = a.node[(size_t)min(t + 8 + u, T - 1) * 256 + tid];
  }
  v4i d0[4], d1[4];
  tile_product(bt[P][0], ctr, b4, d0);
  tile_product(bt[P][1], ctr, b4, d1);
  tile_build1(xs, XS, rtab[P ^ 1][0], bt[P ^ 1][0], tid);
  tile_build1(xs, XS, rtab[P ^ 1][1], bt[P ^ 1][1], tid);
  red[P][0][wave * 4 + g4][r16] = tile_best(d0);  // 16 partial maxima per row, combined by the leaf's wave
  red[P][1][wave * 4 + g4][r16] = tile_best(d1);
  lds_sync();
  // the leaves of trees t and t+1, by waves t mod 4 and t+1 mod 4 (a wave's
  // previous lookup is consumed first)
  const int u = wave - (t & 3);  // (split parts start at multiples of 4 trees)
  if ((u == 0 || (u == 1 && t + 1 < T)) && lane < kTileRows) {
    tile_leaf_consume<KMODE>(a, pend, acc, r0 + lane);
    int col = red[P][u][0][lane];
#pragma unroll
    for (int q = 1; q < 16; ++q) col = max(col, red[P][u][q][lane]);
    col = min(max(col, 0), a.l_pad - 1);  // a valid tree always yields a column in range
    tile_leaf_issue<KMODE>(a, pend, t + u, col);
  }
}

template <int KMODE>
__global__ __launch_bounds__(256) void gemm_tile_kernel(GemmArgs a) {
  constexpr int KMAX = TileLeaf<KMODE>::KMAX;
  extern __shared__ __align__(16) unsigned char smem[];  // feature tile [16][XS], then the waves' partial sums
  __shared__ __align__(16) unsigned char bt[2][2][kTileRows * kTileBStride];
  __shared__ __align__(16) uint2 rtab[2][2][256];
  __shared__ int red[2][2][16][kTileRows];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, r16 = lane & 15;
  // this workgroup's trees [tb, T): all of them unless the trees are split
  const int tb = a.split ? (int)blockIdx.y * a.split : 0;
  const int T = a.split ? min(tb + a.split, a.out.T) : a.out.T;
  const int XS = gemm_tile_xs(a.F);
  float *xs = reinterpret_cast<float *>(smem);
  const int64_t r0 = (int64_t)blockIdx.x * kTileRows;
  if (!a.cols && (a.F & 3) == 0 && (a.Fs & 3) == 0 && (reinterpret_cast<uintptr_t>(a.X) & 15) == 0) {
    // 16-byte loads, four rows' worth in flight before their LDS stores
    const int F4 = a.F >> 2;
#pragma unroll 4
    for (int r = 0; r < kTileRows; ++r) {
      const bool ok = r0 + r < a.n_rows;
      const float4 *src = reinterpret_cast<const float4 *>(a.X + (ok ? r0 + r : (int64_t)0) * a.Fs);
      for (int f = tid; f < F4; f += 256)
        *reinterpret_cast<float4 *>(xs + r * XS + 4 * f) = ok ? src[f] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  } else {
    for (int r = 0; r < kTileRows; ++r) {
      const bool ok = r0 + r < a.n_rows;
      const float *src = a.X + (ok ? r0 + r : (int64_t)0) * a.Fs;
      for (int f = tid; f < a.F; f += 256) xs[r * XS + f] = ok ? xval(src, a.cols, f) : 0.0f;
    }
  }
  // this wave's leaves: A operands (4 C^T) and accumulator biases
  v4i ctr[4][4], b4[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int lt = wave * 4 + j;
    b4[j] = *reinterpret_cast<const v4i *>(a.bias + lt * 16 + 4 * g4);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      ctr[j][kb] = *reinterpret_cast<const v4i *>(a.ct + (size_t)(lt * 16 + r16) * 256 + kb * 64 + 16 * g4);
  }
  // records of trees tb .. tb+3 in LDS, tb+4 .. tb+7 in registers
  uint2 rset[2][2];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    rtab[u >> 1][u & 1][tid] = a.node[(size_t)min(tb + u, T - 1) * 256 + tid];
    rset[u >> 1][u & 1] = a.node[(size_t)min(tb + u + 4, T - 1) * 256 + tid];
  }
  lds_sync();
  tile_build1(xs, XS, rtab[0][0], bt[0][0], tid);
  tile_build1(xs, XS, rtab[0][1], bt[0][1], tid);
  lds_sync();
  double acc[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) acc[k] = 0.0;
  TileLeaf<KMODE> pend;
  for (int t = tb; t < T; t += 4) {
    tile_pair<KMODE, 0>(a, t, xs, XS, bt, rtab, red, rset, ctr, b4, pend, acc, r0, T);
    if (t + 2 < T) tile_pair<KMODE, 1>(a, t + 2, xs, XS, bt, rtab, red, rset, ctr, b4, pend, acc, r0, T);
  }
  if (lane < kTileRows) tile_leaf_consume<KMODE>(a, pend, acc, r0 + lane);
  // partial sums in wave order (the feature tile is no longer read)
  double *part = reinterpret_cast<double *>(smem);
  if (lane < kTileRows) {
#pragma unroll
    for (int k = 0; k < KMAX; ++k) part[(wave * kTileRows + lane) * KMAX + k] = acc[k];
  }
  lds_sync();
  if (wave == 0 && lane < kTileRows && r0 + lane < a.n_rows) {
    double s[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) s[k] = 0.0;
    for (int w = 0; w < 4; ++w) {
#pragma unroll
      for (int k = 0; k < KMAX; ++k) s[k] += part[(w * kTileRows + lane) * KMAX + k];
    }
    if (a.split) {
      double *dst = a.partial + ((size_t)blockIdx.y * a.n_rows + r0 + lane) * a.out.K;
#pragma unroll
      for (int k = 0; k < KMAX; ++k)
        if (k < a.out.K) dst[k] = s[k];
    } else {
      finish_row<KMAX>(a.out, s, r0 + lane);
    }
  }
}

// Wide rows with two groups of four waves on one 16-row feature tile (eight
// waves, two per SIMD, where the four-wave kernel leaves one per SIMD, with
// the predicate build's LDS round trips exposed). Group g takes trees
// tb + g, tb + g + 2, ..., one per step between two barriers: in step k it
// multiplies its tree k (built in step k - 1) and builds its tree k + 1, so
// each wave overlaps its own matrix instructions with LDS reads, and the
// other group's wave on the same SIMD fills its waits. Each group has its
// own double-buffered predicate tile, record table and maxima (1 KiB more
// LDS than the four-wave kernel's pairs). Tree k of a group is looked up by
// the group's wave k mod 4; the eight waves' sums are added in wave order.
constexpr int kTile2Threads = 512;
// Maxima of a tree: per row, the 16 lane groups' values in one 80-byte row
// (the lookup reads a row with four 16-byte loads; the 64 lanes writing at
// once, rows 20 words apart, fall on 64 different banks).
constexpr int kTile2RedStride = 20;

template <int KMODE, int KM, int P>
__device__ __forceinline__ void tile2_step(const GemmArgs &a, int k, int grp, int mine, int tb, int T, const float *xs,
                                           int XS, unsigned char (*bt)[kTileRows * kTileBStride], uint2 (*rtab)[256],
                                           int (*red)[kTileRows][kTile2RedStride], uint2 (&rset)[2],
                                           const v4i (&ctr)[4][4],
                                           const v4i (&b4)[4], TileLeaf<KMODE, KM> &pend, double (&acc)[KM],
                                           int64_t r0) {
  // bt, rtab, red: this group's buffers; group tree k is tree tb + grp + 2k
  const int gt = threadIdx.x & 255, lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) & 3;
  const int g4 = lane >> 4, r16 = lane & 15;
  rtab[P][gt] = rset[P];  // records of group tree k + 2 (loaded two steps ago)
  rset[P] = a.node[(size_t)min(tb + grp + 2 * (k + 4), T - 1) * 256 + gt];
  v4i d[4];
  tile_product(bt[P], ctr, b4, d);
  tile_build1(xs, XS, rtab[P ^ 1], bt[P ^ 1], gt);
  red[P][r16][wave * 4 + g4] = tile_best(d);
  lds_sync();
  if (k < mine && wave == (k & 3)) {
    // the lookup makes this wave the last to reach the next barrier: its
    // instructions go first on its SIMD meanwhile (measured: 5.98 -> 5.84 ms
    // on the 2,000-feature forest; raising the build's priority as well was
    // slower)
    __builtin_amdgcn_s_setprio(2);
    if (lane < kTileRows) {
      tile_leaf_consume(a, pend, acc, r0 + lane);
      const v4i *m = reinterpret_cast<const v4i *>(red[P][lane]);
      const v4i m0 = m[0], m1 = m[1], m2 = m[2], m3 = m[3];
      int col = max(max(hmax4(m0), hmax4(m1)), max(hmax4(m2), hmax4(m3)));
      col = min(max(col, 0), a.l_pad - 1);  // a valid tree always yields a column in range
      tile_leaf_issue(a, pend, tb + grp + 2 * k, col);
    }
    __builtin_amdgcn_s_setprio(0);
  }
}

template <int KMODE, int KM>
__global__ __launch_bounds__(kTile2Threads) void gemm_tile2_kernel(GemmArgs a) {
  constexpr int KMAX = KM;
  extern __shared__ __align__(16) unsigned char smem[];  // feature tile [16][XS], then the waves' partial sums
  __shared__ __align__(16) unsigned char bt[2][2][kTileRows * kTileBStride];  // [group][buffer]
  __shared__ __align__(16) uint2 rtab[2][2][256];
  __shared__ __align__(16) int red[2][2][kTileRows][kTile2RedStride];
  const int tid = threadIdx.x, lane = tid & 63, grp = tid >> 8, gt = tid & 255, wave = (tid >> 6) & 3;
  const int g4 = lane >> 4, r16 = lane & 15;
  const int tb = a.split ? (int)blockIdx.y * a.split : 0;
  const int T = a.split ? min(tb + a.split, a.out.T) : a.out.T;
  const int steps = (T - tb + 1) >> 1;      // group 0's tree count, the larger
  const int mine = (T - tb - grp + 1) >> 1;  // this group's
  const int XS = gemm_tile_xs(a.F);
  float *xs = reinterpret_cast<float *>(smem);
  const int64_t r0 = (int64_t)blockIdx.x * kTileRows;
  if (!a.cols && (a.F & 3) == 0 && (a.Fs & 3) == 0 && (reinterpret_cast<uintptr_t>(a.X) & 15) == 0) {
    const int F4 = a.F >> 2;
#pragma unroll 4
    for (int r = 0; r < kTileRows; ++r) {
      const bool ok = r0 + r < a.n_rows;
      const float4 *src = reinterpret_cast<const float4 *>(a.X + (ok ? r0 + r : (int64_t)0) * a.Fs);
      for (int f = tid; f < F4; f += kTile2Threads)
        *reinterpret_cast<float4 *>(xs + r * XS + 4 * f) = ok ? src[f] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  } else {
    for (int r = 0; r < kTileRows; ++r) {
      const bool ok = r0 + r < a.n_rows;
      const float *src = a.X + (ok ? r0 + r : (int64_t)0) * a.Fs;
      for (int f = tid; f < a.F; f += kTile2Threads) xs[r * XS + f] = ok ? xval(src, a.cols, f) : 0.0f;
    }
  }
  v4i ctr[4][4], b4[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int lt = wave * 4 + j;
    b4[j] = *reinterpret_cast<const v4i *>(a.bias + lt * 16 + 4 * g4);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      ctr[j][kb] = *reinterpret_cast<const v4i *>(a.ct + (size_t)(lt * 16 + r16) * 256 + kb * 64 + 16 * g4);
  }
  // records of group trees 0, 1 in LDS, 2, 3 in registers (trees past the
  // last are clamped to it; their results are not used)
  uint2 rset[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    rtab[grp][u][gt] = a.node[(size_t)min(tb + grp + 2 * u, T - 1) * 256 + gt];
    rset[u] = a.node[(size_t)min(tb + grp + 2 * (u + 2), T - 1) * 256 + gt];
  }
  lds_sync();
  tile_build1(xs, XS, rtab[grp][0], bt[grp][0], gt);
  lds_sync();
  double acc[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) acc[k] = 0.0;
  TileLeaf<KMODE, KM> pend;
  for (int k = 0; k < steps; k += 2) {
    tile2_step<KMODE, KM, 0>(a, k, grp, mine, tb, T, xs, XS, bt[grp], rtab[grp], red[grp], rset, ctr, b4, pend, acc, r0);
    if (k + 1 < steps)
      tile2_step<KMODE, KM, 1>(a, k + 1, grp, mine, tb, T, xs, XS, bt[grp], rtab[grp], red[grp], rset, ctr, b4, pend, acc,
                           r0);
  }
  if (lane < kTileRows) tile_leaf_consume(a, pend, acc, r0 + lane);
  double *part = reinterpret_cast<double *>(smem);
  const int w8 = tid >> 6;
  if (lane < kTileRows) {
#pragma unroll
    for (int k = 0; k < KMAX; ++k) part[(w8 * kTileRows + lane) * KMAX + k] = acc[k];
  }
  lds_sync();
  if (w8 == 0 && lane < kTileRows && r0 + lane < a.n_rows) {
    double s[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) s[k] = 0.0;
    for (int w = 0; w < kTile2Threads / 64; ++w) {
#pragma unroll
      for (int k = 0; k < KMAX; ++k) s[k] += part[(w * kTileRows + lane) * KMAX + k];
    }
    if (a.split) {
      double *dst = a.partial + ((size_t)blockIdx.y * a.n_rows + r0 + lane) * a.out.K;
#pragma unroll
      for (int k = 0; k < KMAX; ++k)
        if (k < a.out.K) dst[k] = s[k];
    } else {
      finish_row<KMAX>(a.out, s, r0 + lane);
    }
  }
}

// ---------------------------------------------------------------------------
// Narrow rows, large batches: 64-row bands. A band's feature tile is small
// (64 x F floats), so three workgroups share a CU. Wave w keeps the A
// operands of leaves 64 w .. 64 w + 63 in registers (as the 16-row tiles do)
// and builds, one tree ahead, the predicate bytes of nodes 64 w .. 64 w + 63
// for all 64 rows of the band (lane = row): a node's record is the same for
// the whole wave, the feature reads of a node are 64 consecutive floats of
// its column, and each lane stores whole 16-byte pieces of its row. The four
// waves then multiply all four 16-row tiles by their leaves, leave per row
// and lane group the maximum over their leaves in LDS, and after the one
// barrier per tree wave t mod 4 picks each row's leaf of tree t from the 16
// maxima. Each wave adds the leaves of its trees in tree order and the four
// waves' sums are added in wave order at the end.
constexpr int kBandRows = 64;
constexpr int kBandXS = kBandRows;  // floats per feature column of the tile
// Predicate tile: row r holds 16 pieces of 16 bytes (nodes 16 p .. 16 p + 15
// in piece p ^ (r mod 16)), so the 16 rows a lane group reads for one piece,
// and the pieces the 64 rows write at once, fall on distinct banks.
__device__ __forceinline__ int band_piece(int r, int p) { return r * 256 + 16 * (p ^ (r & 15)); }

template <int KMODE, int KM>
struct BandLeaf {
  int t = -1;  // tree of the pending lookup, -1 none
  int cls = 0;
  int32_t id = 0;
  float v[KMODE == 2 ? KM : 1];
};

// Predicate bytes (64 where x < threshold, else 0) of nodes 64 w + 16 q ..
// + 15 of tree tn for row `lane` of the band. The records are the same for
// the whole wave and come by vector loads (one address for all lanes):
// scalar loads were slower, as waiting for them also waits for every LDS
// read in flight.
typedef const uint2 *BandRecs;
__device__ __forceinline__ void band_build_q(BandRecs rec, int q, const float *xs, unsigned char *dst, int wave,
                                             int lane) {
  uint2 r[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) r[i] = rec[q * 16 + i];
  float x[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] = xs[r[i].y * kBandXS + lane];
  u32x4 w;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t word = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) word |= (x[j * 4 + b] < as_float(r[j * 4 + b].x) ? 0x40u : 0u) << (8 * b);
    w[j] = word;
  }
  *reinterpret_cast<u32x4 *>(dst + band_piece(lane, wave * 4 + q)) = w;
}

__device__ __forceinline__ BandRecs band_recs(const GemmArgs &a, int tn, int wave) {
  return a.node + (size_t)tn * a.k_pad + wave * 64;
}

template <int KMODE, int KM>
__device__ __forceinline__ void band_consume(const GemmArgs &a, BandLeaf<KMODE, KM> &p, double (&acc)[KM],
                                             int64_t row) {
  if (p.t < 0) return;
  if (KMODE == 2) {
#pragma unroll
    for (int k = 0; k < KM; ++k) acc[k] += (double)p.v[k];
  } else if (KMODE == 0) {
    acc[0] += (double)p.v[0];
  } else {
#pragma unroll
    for (int k = 0; k < KM; ++k)
      if (k == p.cls) acc[k] += (double)p.v[0];
  }
  if (a.leaf_ids && row < a.n_rows) a.leaf_ids[row * a.out.T + p.t] = p.id;
  p.t = -1;
}

template <int KMODE, int KM>
__global__ __launch_bounds__(256) void gemm_band_kernel(GemmArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];  // feature tile [F][kBandXS]
  __shared__ __align__(16) unsigned char bt[2][kBandRows * 256];
  // per row, the 16 lane groups' maxima clamped to [-1, 255] (only a column
  // that is not negative is a match)
  __shared__ __align__(16) short red[2][kBandRows][16];
  static_assert((size_t)4 * kBandRows * HB_MAX_OUTPUTS * 8 <= sizeof(bt), "partial sums reuse the predicate tiles");
  const int tid = threadIdx.x, lane = tid & 63, g4 = lane >> 4, r16 = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.out.T;
  float *xs = reinterpret_cast<float *>(smem);
  const int64_t r0 = (int64_t)blockIdx.x * kBandRows;
  const int64_t row = r0 + lane;
  for (int e = tid; e < kBandRows * a.F; e += 256) {
    const int r = e / a.F, f = e - r * a.F;
    xs[f * kBandXS + r] = r0 + r < a.n_rows ? xval(a.X + (r0 + r) * a.Fs, a.cols, f) : 0.0f;
  }
  v4i ctr[4][4], b4[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int lt = wave * 4 + j;
    b4[j] = *reinterpret_cast<const v4i *>(a.bias + lt * 16 + 4 * g4);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      ctr[j][kb] = *reinterpret_cast<const v4i *>(a.ct + (size_t)(lt * 16 + r16) * 256 + kb * 64 + 16 * g4);
  }
  lds_sync();
#pragma unroll
  for (int q = 0; q < 4; ++q) band_build_q(band_recs(a, 0, wave), q, xs, bt[0], wave, lane);
  lds_sync();
  double acc[KM];
#pragma unroll
  for (int k = 0; k < KM; ++k) acc[k] = 0.0;
  BandLeaf<KMODE, KM> pend;
  for (int t = 0; t < T; ++t) {
    const int P = t & 1;
    const BandRecs next = band_recs(a, min(t + 1, T - 1), wave);
    // tree t's products, 16 rows at a time, each row tile's four leaf tiles
    // as four independent chains; per row and lane group the maximum over
    // this wave's leaves (the selected leaf's column, or a negative value).
    // Then tree t+1's predicate operand (building it between the row tiles
    // was slower).
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      v4i bop[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        bop[kb] = *reinterpret_cast<const v4i *>(bt[P] + band_piece(16 * rt + r16, kb * 4 + g4));
      v4i d[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          d[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ctr[j][kb], bop[kb], kb ? d[j] : b4[j], 0, 0, 0);
      const int best = max(max(hmax4(d[0]), hmax4(d[1])), max(hmax4(d[2]), hmax4(d[3])));
      red[P][16 * rt + r16][wave * 4 + g4] = (short)min(max(best, -1), 255);
    }
    if (t + 1 < T) {
#pragma unroll
      for (int q = 0; q < 4; ++q) band_build_q(next, q, xs, bt[P ^ 1], wave, lane);
    }
    lds_sync();
    if (wave == (t & 3)) {
      band_consume<KMODE, KM>(a, pend, acc, row);
      int col = -1;
#pragma unroll
      for (int i = 0; i < 16; ++i) col = max(col, (int)red[P][lane][i]);
      col = min(max(col, 0), a.l_pad - 1);  // a valid tree always yields a column in range
      const size_t lrec = (size_t)t * a.l_pad + (size_t)col;
      pend.t = t;
      pend.id = a.leaf_id[lrec];
      if (KMODE == 2) {
#pragma unroll
        for (int k = 0; k < KM; ++k) pend.v[k] = k < a.LD ? a.leaf_value[lrec * a.LD + k] : 0.0f;
      } else {
        pend.v[0] = a.leaf_value[lrec];
        if (KMODE == 1) pend.cls = a.tree_class[t];
      }
    }
  }
  band_consume<KMODE, KM>(a, pend, acc, row);
  // the four waves' sums in wave order (the predicate tiles are no longer read)
  double *part = reinterpret_cast<double *>(&bt[0][0]);
#pragma unroll
  for (int k = 0; k < KM; ++k) part[(wave * kBandRows + lane) * KM + k] = acc[k];
  lds_sync();
  if (wave == 0 && row < a.n_rows) {
    double s[KM];
#pragma unroll
    for (int k = 0; k < KM; ++k) s[k] = 0.0;
    for (int w = 0; w < 4; ++w) {
#pragma unroll
      for (int k = 0; k < KM; ++k) s[k] += part[(w * kBandRows + lane) * KM + k];
    }
    finish_row<KM>(a.out, s, row);
  }
}

using GemmFn = void (*)(GemmArgs);

template <int KB, bool CT, bool XL, int ROWS, bool COLS = false>
GemmFn pick_mode(int kmode) {
  if (kmode == 0) return gemm_kernel<KB, CT, XL, 0, ROWS, COLS>;
  if (kmode == 1) return gemm_kernel<KB, CT, XL, 1, ROWS, COLS>;
  return gemm_kernel<KB, CT, XL, 2, ROWS, COLS>;
}

// cols: features read straight from global memory go through the column list
template <int KB>
GemmFn pick_gemm(bool ct, bool xl, int kmode, int rows, bool cols) {
  if (rows == 512) return ct && xl ? pick_mode<KB, true, true, 512>(kmode) : nullptr;
  if (xl) return ct ? pick_mode<KB, true, true, 256>(kmode) : pick_mode<KB, false, true, 256>(kmode);
  if (ct) return cols ? pick_mode<KB, true, false, 256, true>(kmode) : pick_mode<KB, true, false, 256>(kmode);
  return cols ? pick_mode<KB, false, false, 256, true>(kmode) : pick_mode<KB, false, false, 256>(kmode);
}

}  // namespace

// Batches from three 64-row bands per CU up take the band kernel.
constexpr int64_t kBandMinRows = 3 * 256 * kBandRows;

static GemmFn band_fn(int kmode, int width) {
  if (kmode == 0) return gemm_band_kernel<0, 1>;
  if (kmode == 1) return width <= 8 ? gemm_band_kernel<1, 8> : gemm_band_kernel<1, 16>;
  return width <= 2 ? gemm_band_kernel<2, 2> : width <= 8 ? gemm_band_kernel<2, 8> : gemm_band_kernel<2, 16>;
}

int launch_gemm(const EnsembleDev &e, const GemmDev &t, const float *X, int64_t n_rows, float *scores,
                int32_t *leaf_ids, const Launch &L, hipStream_t stream, std::string *err) {
  if (!t.node || !t.shape || !t.ct || !t.bias || !t.leaf_value || !t.leaf_id) {
    *err = "GEMM tables missing";
    return HB_ERR_INVALID_ARG;
  }
  if (t.k_pad % 64 || t.k_pad < 64 || t.k_pad > 256 || t.l_pad % 16 || t.l_pad < 16 || t.l_pad > 256) {
    *err = "GEMM tables have an unexpected shape";
    return HB_ERR_INVALID_ARG;
  }
  if (n_rows <= 0) return HB_OK;
  int dev = 0, lds_max = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) {
    *err = "hipDeviceGetAttribute failed";
    return HB_ERR_HIP;
  }
  const size_t nodes = 2 * (size_t)kTG * node_lds_bytes(t.k_pad);
  const size_t ct_bytes = (size_t)t.l_pad * (t.k_pad + kCtPad) + (size_t)t.l_pad * 4;
  auto x_bytes = [&](int rows) { return ((size_t)e.n_cols * (rows + 8) * 4 + 15) / 16 * 16; };
  auto stage_bytes = [&](int rows) { return (size_t)(rows / 64) * 16 * (kIdGroup / 4) * 16; };
  const bool ct = t.n_shapes == 1 && ct_bytes + nodes + stage_bytes(256) <= (size_t)lds_max;
  int rows = 256;
  if (ct && n_rows >= 64 * 512 && ct_bytes + nodes + x_bytes(512) + stage_bytes(512) <= (size_t)lds_max) rows = 512;
  const bool xl = (ct ? ct_bytes : 0) + nodes + x_bytes(rows) + stage_bytes(rows) <= (size_t)lds_max;
  size_t dyn = (xl ? x_bytes(rows) : 0) + (ct ? ct_bytes : 0) + nodes;
  if (dyn + stage_bytes(rows) > (size_t)lds_max) {
    *err = "GEMM node tables do not fit in LDS";
    return HB_ERR_UNSUPPORTED;
  }
  const int kmode = e.leaf_dim > 1 ? 2 : (e.n_outputs > 1 ? 1 : 0);
  const int kb = t.k_pad / 64;
  const bool cols = e.cols != nullptr;
  GemmFn fn = kb == 1 ? pick_gemm<1>(ct, xl, kmode, rows, cols)
              : kb == 2 ? pick_gemm<2>(ct, xl, kmode, rows, cols)
              : kb == 3 ? pick_gemm<3>(ct, xl, kmode, rows, cols)
                        : pick_gemm<4>(ct, xl, kmode, rows, cols);
  int threads = rows;
  std::string name = "gemm_kernel<" + std::to_string(kb) + ", " + (ct ? "true" : "false") + ", " +
                     (xl ? "true" : "false") + ", " + std::to_string(kmode) + ", " + std::to_string(rows) + ", " +
                     (cols && !xl ? "true" : "false") + ">";
  bool piped = false, tile_wide = false;
  if (rows == 512 && ct && xl && kb == 4 && t.l_pad == 256) {
    // the software-pipelined kernel needs no node chunks; it runs only with
    // 512-row workgroups (two waves per SIMD), since wherever a 256-row
    // pipelined workgroup would fit, the 16-row tiles below fit too
    const size_t need = x_bytes(rows) + ct_bytes;
    if (need + stage_bytes(rows) <= (size_t)lds_max) {
      fn = kmode == 0 ? gemm_pipe_kernel<0, 512> : kmode == 1 ? gemm_pipe_kernel<1, 512> : gemm_pipe_kernel<2, 512>;
      name = "gemm_pipe_kernel<" + std::to_string(kmode) + ", 512>";
      dyn = need;
      piped = true;
    }
  }
  bool banded = false;
  if (!piped && t.n_shapes == 1 && kb == 4 && t.l_pad == 256 && n_rows >= kBandMinRows) {
    // 64-row bands where three of them fit a CU's LDS (narrow rows)
    const size_t band_dyn = (size_t)e.n_cols * kBandXS * 4;
    const size_t band_static = (size_t)2 * kBandRows * 256 + (size_t)2 * kBandRows * 16 * 2;
    if (3 * (band_dyn + band_static) <= (size_t)lds_max) {
      fn = band_fn(kmode, kmode == 2 ? e.leaf_dim : e.n_outputs);
      dyn = band_dyn;
      rows = kBandRows;
      threads = 256;
      banded = true;
      name = std::string("gemm_band_kernel<") + std::to_string(kmode) + ", " +
             std::to_string(kmode == 0 ? 1 : (kmode == 2 && e.leaf_dim <= 2) ? 2 : (kmode == 2 ? e.leaf_dim : e.n_outputs) <= 8 ? 8 : 16) + ">";
    }
  }
  if (!piped && !banded && t.n_shapes == 1 && kb == 4 && t.l_pad == 256) {
    // 16-row tiles with C^T in registers, unless the pipelined kernel gets
    // 512-row workgroups (two waves per SIMD): wide rows, where its feature
    // tile does not fit, and 256-row workgroups, one wave per SIMD (measured:
    // 7 x 500 trees over 54 features at 1M rows 413 -> 361 ms; the 500-tree
    // 28-feature model stays on 512-row pipelined workgroups, 28 against 39 ms)
    const int kmax = kmode == 0 ? 1 : HB_MAX_OUTPUTS;
    const size_t tile_dyn = std::max((size_t)kTileRows * gemm_tile_xs(e.n_cols) * 4, (size_t)4 * kTileRows * kmax * 8);
    const size_t tile_static = (size_t)4 * kTileRows * kTileBStride + 4 * 256 * 8 + 4 * 16 * kTileRows * 4;
    if (tile_dyn + tile_static <= (size_t)lds_max) {
      const bool wide = 2 * (tile_dyn + tile_static) > (size_t)lds_max;  // one workgroup per CU
      tile_wide = wide;
      // one workgroup per CU: eight waves in two groups on the one feature
      // tile (the same static LDS; the eight waves' partial sums in the tile
      // at the end, which a tile this wide always holds)
      const size_t tile2_dyn = std::max(tile_dyn, (size_t)8 * kTileRows * kmax * 8);
      const size_t tile2_static = (size_t)4 * kTileRows * kTileBStride + 4 * 256 * 8 + 4 * kTileRows * kTile2RedStride * 4;
      if (!wide) {
        fn = kmode == 0 ? gemm_tile_kernel<0> : kmode == 1 ? gemm_tile_kernel<1> : gemm_tile_kernel<2>;
        dyn = tile_dyn;
        threads = 256;
        name = "gemm_tile_kernel<" + std::to_string(kmode) + ">";
      } else if (tile2_dyn + tile2_static <= (size_t)lds_max) {
        const int width = kmode == 2 ? e.leaf_dim : e.n_outputs;
        const int km = kmode == 0 ? 1 : kmode == 2 && width <= 2 ? 2 : width <= 8 ? 8 : HB_MAX_OUTPUTS;
        fn = kmode == 0    ? gemm_tile2_kernel<0, 1>
             : kmode == 1  ? (km == 8 ? gemm_tile2_kernel<1, 8> : gemm_tile2_kernel<1, HB_MAX_OUTPUTS>)
             : km == 2     ? gemm_tile2_kernel<2, 2>
             : km == 8     ? gemm_tile2_kernel<2, 8>
                           : gemm_tile2_kernel<2, HB_MAX_OUTPUTS>;
        dyn = tile2_dyn;
        threads = kTile2Threads;
        name = "gemm_tile2_kernel<" + std::to_string(kmode) + ", " + std::to_string(km) + ">";
      }
      rows = kTileRows;
    }
  }
  if (!fn) {
    *err = "no GEMM kernel for this configuration";
    return HB_ERR_UNSUPPORTED;
  }
  GemmArgs a{};
  a.X = X;
  a.n_rows = n_rows;
  a.F = e.n_cols;
  a.Fs = e.n_features;
  a.cols = e.cols;
  a.leaf_ids = leaf_ids;
  a.out = OutArgs{scores, e.n_trees, e.n_outputs, e.aggregation, e.transform, e.base_score};
  a.tree_class = e.tree_class;
  a.LD = e.leaf_dim;
  a.node = t.node;
  a.shape = t.shape;
  a.ct = t.ct;
  a.bias = t.bias;
  a.leaf_value = t.leaf_value;
  a.leaf_id = t.leaf_id;
  a.k_pad = t.k_pad;
  a.l_pad = t.l_pad;
  a.ids_vec = (e.n_trees % 4 == 0) && ((reinterpret_cast<uintptr_t>(leaf_ids) & 15) == 0);
  const int64_t blocks = (n_rows + rows - 1) / rows;
  // Small batch with a workspace on the 16-row tiles: divide the trees, in
  // groups of 4, among `parts` workgroups per tile (a batch of a few tiles
  // otherwise walks every tree on a few CUs), then add the partial sums in
  // a fixed order. With `resident` tile workgroups at once the call takes
  // about ceil(parts x tiles / resident) rounds of `per` groups each plus a
  // fixed cost per workgroup (C^T, feature tile) worth about
  // kTileOverheadGroups groups; take the fewest parts reaching the least.
  int split = 1;
  if (rows == kTileRows && L.ptr && n_rows <= kGemmSplitMaxRows) {
    const int64_t groups = (e.n_trees + kGemmSplitGroup - 1) / kGemmSplitGroup;
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) {
      *err = "hipDeviceGetAttribute(MultiprocessorCount) failed";
      return HB_ERR_HIP;
    }
    const int64_t resident = (int64_t)cus * (tile_wide ? 1 : 2);
    const int64_t row_bytes = n_rows * e.n_outputs * 8;
    constexpr int64_t kTileOverheadGroups = 8;
    int64_t best_cost = (blocks + resident - 1) / resident * (groups + kTileOverheadGroups), best_per = groups;
    for (int64_t p = 2; p <= groups; ++p) {
      const int64_t per = (groups + p - 1) / p, parts = (groups + per - 1) / per;
      if (parts * row_bytes > L.bytes) break;
      const int64_t cost = (parts * blocks + resident - 1) / resident * (per + kTileOverheadGroups);
      if (cost < best_cost) {
        best_cost = cost;
        best_per = per;
      }
    }
    if (best_per < groups) {
      split = (int)((groups + best_per - 1) / best_per);
      a.split = (int)best_per * kGemmSplitGroup;
      a.partial = static_cast<double *>(L.ptr);
    }
  }
  if (L.plan) {
    plan_line(L.plan, name, blocks, split, threads, dyn);
    if (split > 1) return split_finish(nullptr, split, n_rows, a.out, L.plan, stream, err);
    return HB_OK;
  }
  hipError_t rc = hipFuncSetAttribute(reinterpret_cast<const void *>(fn),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (rc != hipSuccess) {
    *err = std::string("hipFuncSetAttribute: ") + hipGetErrorString(rc);
    return HB_ERR_HIP;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)blocks, (unsigned)split), dim3(threads), dyn, stream, a);
  rc = hipGetLastError();
  if (rc != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(rc);
    return HB_ERR_HIP;
  }
  if (split > 1) return split_finish(a.partial, split, n_rows, a.out, nullptr, stream, err);
  return HB_OK;
}

}  // namespace hb
