// hb_fast.h -- the fast traversal kernel template (see the comment below);
// included by the hb_fast_{ptt,tt}_<rows>.hip units, which instantiate it.
#pragma once

#include <type_traits>

#include "hb_device.h"

namespace hb {
namespace {

// ---------------------------------------------------------------------------
// Fast traversal kernels for scalar leaves and inputs whose feature tile fits
// in LDS. Differences from traverse_kernel:
//   * each tree owns one packed block (node records, then leaf records
//     {value, caller id}); chunks of TC consecutive blocks pass through LDS:
//     chunk c+1 is loaded into registers before chunk c is walked and stored
//     to LDS after it (into the other buffer when double-buffered), so the
//     load latency hides behind the walk;
//   * trees of a chunk and levels are fully unrolled with compile-time LDS
//     offsets, and the walk state is the byte offset of the current record;
//   * PTT: heap index a lives as s = 8a; the child is 2s + 8*(x >= t) and,
//     after D steps, s is exactly the offset of the leaf record (leaves follow
//     the 2^D node slots);
//   * TT: a node record {threshold, feature | 8 * right << 16} (children are
//     adjacent, left = right - 1) makes a step one shift and one subtract of
//     8 or 0; a leaf holds threshold -inf and points to itself;
//   * multi-output: the output column of each tree is uniform across a wave,
//     so the per-row double accumulators are updated by register index (the
//     columns of a chunk are loaded one chunk ahead, lane g holding tree g's);
//     vector leaves add every value of the reached leaf, read from the
//     strategy's leaf-value table in global memory (L2-resident).

// Barrier for LDS traffic only: orders this workgroup's LDS accesses across
// the barrier without waiting for outstanding global stores (the leaf-id
// writes keep draining while the next chunk is walked).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// One chunk of tree blocks held in registers between its global load (issued
// before the current chunk is walked) and its LDS store (after the walk).
// Native vector words (not the HIP uint4 struct) so they stay in VGPRs.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int ROWS, int N16>
struct ChunkPrefetch {
  static constexpr int PER = (N16 + ROWS - 1) / ROWS;
  u32x4 v[PER];
  // every lane loads (a clamped, in-bounds index)
  __device__ __forceinline__ void load(const uint4 *__restrict__ src) {
    const u32x4 *s = reinterpret_cast<const u32x4 *>(src);
#pragma unroll
    for (int i = 0; i < PER; ++i) v[i] = s[min(i * ROWS + (int)threadIdx.x, N16 - 1)];
  }
  __device__ __forceinline__ void store(uint4 *dst) const {
    u32x4 *d = reinterpret_cast<u32x4 *>(dst);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = i * ROWS + (int)threadIdx.x;
      if (u < N16) d[u] = v[i];
    }
  }
};

template <int MODE>
constexpr int kFastMaxLgFor = MODE == 0 ? 10 : MODE == 3 ? 8 : 11;

struct IdPack;
struct IdPack8;

template <int MODE, int LG, int KM, int ROWS, int BUDGET>
struct FastCfg {
  static constexpr int TB = fast_tree_bytes(MODE, LG);
  static constexpr int TC = fast_tc_m(MODE, TB, BUDGET);
  static constexpr int BUFS = fast_bufs_m(MODE, TB, BUDGET);
  static constexpr int CPF = kFastIdGroup / TC;  // chunks per leaf-id flush
  static constexpr int CHUNK16 = TC * TB / 16;
  static constexpr int KMAX = KM;  // accumulators: 1, 2 or HB_MAX_OUTPUTS
  static constexpr bool MULTI = KM > 1;
  // two outputs: the chunk's 2-vector leaves are held in registers for one
  // walk (up to 8 trees per chunk; larger chunks add them at once)
  static constexpr bool VHOLD = KM == 2 && TC <= 8;
  static constexpr int VH = VHOLD ? TC : 1;
  // TT leaf records in global memory (mode 2), one output, chunks of up to 8
  // trees: the records are held in registers for one walk, and the chunk's
  // leaf ids and sums are taken one chunk late
  static constexpr bool LAG = MODE == 2 && KM == 1 && TC <= 8;
  static constexpr int LH = LAG ? TC : 1;
  // chunks of 8 trees: the leaf-id lines that end inside the chunk (at its
  // fourth tree) leave at the start of the next chunk, with those that end
  // at its last tree, and the ids of its last four trees wait in two
  // registers until then (their slots still hold ids those lines need)
  static constexpr bool DEFER = TC == 8;
  // PTT with the leaf values in global memory (mode 3): the values are read
  // right after the walk and added after the next one, so their latency
  // hides behind a walk; the ids are the leaves' slots, held as bytes
  static constexpr bool GV = MODE == 3;
  static constexpr int GVH = GV ? TC : 1;
  // several outputs (one per tree class): the output column of each held
  // value, wave-uniform
  static constexpr int GKH = GV && MULTI ? TC : 1;
  using Pack = typename std::conditional<GV, IdPack8, IdPack>::type;
};

// Leaf ids of a 32-tree group, one row per lane, as 16-bit halves: tree q of
// the group sits in bits 16 (q & 1) of dword (q >> 1) & 3 of quad q >> 3.
// pend holds the ids of trees 4..7 of a chunk of 8 until they may take their
// slots (same halves: trees 4 and 5 in pend[0], 6 and 7 in pend[1]).
constexpr int kIdQuads = kFastIdGroup / 8;
struct IdPack {
  u32x4 q[kIdQuads];
  uint32_t pend[2];
  __device__ __forceinline__ u32x4 &operator[](int j) { return q[j]; }
  __device__ __forceinline__ const u32x4 &operator[](int j) const { return q[j]; }
};

// q is a constant once the chunk loop is unrolled
__device__ __forceinline__ void put_id(IdPack &ids, int q, uint32_t id) {
  if (q & 1)
    ids[q >> 3][(q >> 1) & 3] |= id << 16;
  else
    ids[q >> 3][(q >> 1) & 3] = id;
}
// tree g in 4..7 of a chunk of 8, held until its slot is free
__device__ __forceinline__ void hold_id(IdPack &ids, int g, uint32_t id) {
  if (g & 1)
    ids.pend[(g - 4) >> 1] |= id << 16;
  else
    ids.pend[(g - 4) >> 1] = id;
}
template <int QX>
__device__ __forceinline__ void put_pending(IdPack &ids) {
  ids[QX][2] = ids.pend[0];
  ids[QX][3] = ids.pend[1];
}

// Leaf slots of a 32-tree group as bytes, for PTT trees of depth <= 8 whose
// caller ids are the slot plus one base (heap-ordered perfect trees: the
// leaves follow the 2^D - 1 decision nodes); the ids are formed as they
// leave. Tree q of the group sits in byte q & 3 of dword q >> 2 (component
// (q >> 2) & 3 of quad q >> 4); pend holds trees 4..7 of a chunk of 8, the
// whole dword their slots take. Half the registers and half the staging of
// 16-bit ids.
struct IdPack8 {
  u32x4 q[2];
  uint32_t pend;
};
__device__ __forceinline__ void put_id(IdPack8 &ids, int q, uint32_t slot) {
  const int d = q >> 2;
  if ((q & 3) == 0)
    ids.q[d >> 2][d & 3] = slot;
  else
    ids.q[d >> 2][d & 3] |= slot << (8 * (q & 3));
}
__device__ __forceinline__ void hold_id(IdPack8 &ids, int g, uint32_t slot) {
  if (g == 4)
    ids.pend = slot;
  else
    ids.pend |= slot << (8 * (g - 4));
}
template <int QX>
__device__ __forceinline__ void put_pending(IdPack8 &ids) {
  ids.q[(2 * QX + 1) >> 2][(2 * QX + 1) & 3] = ids.pend;
}

// Leaf ids leave in whole 128-byte lines of the output, each as soon as its
// last tree is walked. Row r's ids start at int offset b + r T (b: the
// output's offset within a line, in ints), so row r's lines begin at trees
// congruent to phi(r) = -(b + r T) mod 32; with T a multiple of 4 and a
// 16-byte aligned output, phi is a multiple of 4 that depends on r mod 8
// only, and byte k of id_phase lists the residues r mod 8 whose lines begin
// at trees congruent to 4k. After every fourth tree the lanes of the rows
// whose line just ended hand its 32 ids (the last 32 slots of their IdPack)
// to the whole wave through a 512-byte staging area, and one store
// instruction writes the eight lines (lines that end with a chunk leave at
// the start of the next one, once its prefetch is issued, since a load
// issued behind a store is only usable once the store is acknowledged:
// vmcnt retires both in issue order). For the usual tree counts only one
// residue in eight has a line ending at a given tree, so the stores spread
// evenly over the walk instead of leaving in bursts, and each line reaches
// memory whole.
struct IdOut {
  bool on;            // leaf ids requested and the row layout allows vector stores (uniform)
  u32x4 *stage;       // this wave's staging area: two lines of 8 rows x 64 bytes
  int64_t r0w;        // first row of the wave
  int t_begin;        // first tree of this workgroup's part
  uint32_t id_base;   // IdPack8: caller id of leaf slot 0
  // IdPack8 two-line passes, per lane (i = lane / 8, k = lane % 8): 4 k,
  // 32 i, and the byte offset (8 i T + 4 k) 4 of the four ids it stores
  uint32_t k4, i32, goff;
};

template <int ROWS>
__device__ __forceinline__ IdOut make_id_out(bool on, u32x4 *stage, int t_begin, uint32_t id_base, int T) {
  // the wave's first row is uniform: keep it (and the per-pass row and tree
  // offsets computed from it) in scalar registers
  const int64_t r0w = (int64_t)blockIdx.x * ROWS + 64 * __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t k4 = 4u * (lane & 7u), i8 = lane & ~7u;
  return IdOut{on, stage, r0w, t_begin, id_base, k4, 4u * i8, 4u * (i8 * (uint32_t)T + k4)};
}

// Writes, for the rows of residue rho in this wave, the ids of trees
// [max(lo, t_end - 31), min(t_end, T - 1)]; c = (t_end + 1) mod 32 is the
// slot of tree t_end - 31. lo and T are multiples of 4, and so is t_end + 1.
__device__ __forceinline__ void id_pass(int32_t *leaf_ids, int64_t n_rows, int T, const IdOut &io,
                                        const IdPack &ids, int rho, int t_end, int c, int lo) {
  // as a reader, lane (i = lane / 8, k = lane % 8) stores ids 4k .. 4k+3 of
  // row i of the pass; the per-lane offsets are recomputed here rather than
  // held in registers across the walk
  const int lane = threadIdx.x & 63;
  const int k4 = 4 * (lane & 7), row8 = lane & ~7;  // 4 k, 8 i
  if (k4 == 4 * rho) {
    // quad j of row i at slot (j + i / 2) mod 4: the eight writers touch distinct banks
    const int i = (threadIdx.x & 63) >> 3;
#pragma unroll
    for (int j = 0; j < kIdQuads; ++j) io.stage[i * kIdQuads + ((j + (i >> 1)) & 3)] = ids[j];
  }
  __builtin_amdgcn_wave_barrier();
  // ids 2 slot .. of row i sit at byte 2 slot of its staged row, rotated by 16 (i / 2)
  const int rd = 2 * k4 + (row8 & ~15);  // 8 k + 16 (i / 2)
  const uint2 v = *reinterpret_cast<const uint2 *>(reinterpret_cast<const unsigned char *>(io.stage) + 8 * row8 +
                                                   ((2 * c + rd) & 63));
  const int64_t row0 = io.r0w + rho;
  const int rem = (int)min(n_rows - row0, (int64_t)64);
  const int tb = t_end - 31;
  if (row8 < rem && k4 >= lo - tb && k4 < T - tb) {
    int32_t *dst = leaf_ids + (row0 * T + tb) + ((uint32_t)row8 * (uint32_t)T + (uint32_t)k4);
    const i32x4 o{(int)(v.x & 0xffffu), (int)(v.x >> 16), (int)(v.y & 0xffffu), (int)(v.y >> 16)};
    // streaming: whole lines need no merging in L2, and allocating them
    // there would evict the blocks other workgroups are about to stage
    __builtin_nontemporal_store(o, reinterpret_cast<i32x4 *>(dst));
  }
  __builtin_amdgcn_wave_barrier();
}

// id_pass for 8-bit slots: a staged row is 32 bytes (two quads, the eight
// writers of one instruction 32 bytes apart: distinct banks); a reader takes
// the four slots of its ids in one dword and adds the base.
__device__ __forceinline__ void id_pass(int32_t *leaf_ids, int64_t n_rows, int T, const IdOut &io,
                                        const IdPack8 &ids, int rho, int t_end, int c, int lo) {
  const int lane = threadIdx.x & 63;
  const int k4 = 4 * (lane & 7), i = lane >> 3;
  if (k4 == 4 * rho) {
    io.stage[2 * i] = ids.q[0];
    io.stage[2 * i + 1] = ids.q[1];
  }
  __builtin_amdgcn_wave_barrier();
  const uint32_t v =
      *reinterpret_cast<const uint32_t *>(reinterpret_cast<const unsigned char *>(io.stage) + 32 * i + ((c + k4) & 31));
  const int64_t row0 = io.r0w + rho;
  const int rem = (int)min(n_rows - row0, (int64_t)64);
  const int tb = t_end - 31;
  if (8 * i < rem && k4 >= lo - tb && k4 < T - tb) {
    int32_t *dst = leaf_ids + (row0 * T + tb) + ((uint32_t)(8 * i) * (uint32_t)T + (uint32_t)k4);
    const uint32_t b = io.id_base;
    const i32x4 o{(int)(b + (v & 0xffu)), (int)(b + ((v >> 8) & 0xffu)), (int)(b + ((v >> 16) & 0xffu)),
                  (int)(b + (v >> 24))};
    __builtin_nontemporal_store(o, reinterpret_cast<i32x4 *>(dst));
  }
  __builtin_amdgcn_wave_barrier();
}

// The lane's index in its wave, read afresh at each use: the compiler cannot
// hoist it, or the per-lane offsets derived from it, out of the tree loop
// (held across the walk they would take the registers the walk needs).
__device__ __forceinline__ int lane_fresh() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Two lines per row group at once (chunks of 8 trees, one residue ending a
// line at each of the chunk's two line trees): the rows of residue rho0,
// whose line ended at tree te0 (the chunk's fourth tree), stage the pack as
// it stood then (quad QX's upper half still holding the ids of 32 trees
// earlier), the rows of rho1 (line ended at te1, the chunk's last tree) stage
// it with that half from pend; the 16 writers of one instruction touch
// distinct banks (row i of line r is rotated by ((i / 4) + 2 r) mod 4
// quads). Then every lane stores four ids of one row of each line. The two
// staged lines take the wave's two 512-byte staging halves; a write of 8 or
// 16 lanes costs the LDS as much as one of 64, so this halves the staging
// writes of two separate passes.
template <int QX>
__device__ __forceinline__ void id_pass2(int32_t *leaf_ids, int64_t n_rows, int T, const IdOut &io, const IdPack &ids,
                                         int rho0, int te0, int c0, int rho1, int te1, int c1, int lo) {
  const int lane = lane_fresh();
  const int k = lane & 7, i = lane >> 3;
  if (k == rho0 || k == rho1) {
    const int r = k == rho1 ? 1 : 0;
    const int rot = ((i >> 2) + 2 * r) & 3;
    u32x4 *dst = io.stage + r * (8 * kIdQuads) + i * kIdQuads;
#pragma unroll
    for (int j = 0; j < kIdQuads; ++j) {
      u32x4 q = ids[j];
      if (j == QX) {
        q[2] = r ? ids.pend[0] : q[2];
        q[3] = r ? ids.pend[1] : q[3];
      }
      dst[(j + rot) & 3] = q;
    }
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int c = r ? c1 : c0;
    const int rot = ((i >> 2) + 2 * r) & 3;
    // ids 2 slot .. of row i of line r sit at byte 2 slot of its staged row, rotated by 16 rot
    const uint2 v = *reinterpret_cast<const uint2 *>(reinterpret_cast<const unsigned char *>(io.stage) + 512 * r +
                                                     64 * i + ((2 * c + 8 * k + 16 * rot) & 63));
    const int64_t row0 = io.r0w + (r ? rho1 : rho0);
    const int rem = (int)min(n_rows - row0, (int64_t)64);
    const int tb = (r ? te1 : te0) - 31;
    const int k4 = 4 * k;
    if (8 * i < rem && k4 >= lo - tb && k4 < T - tb) {
      int32_t *dst = leaf_ids + (row0 * T + tb) + ((uint32_t)(8 * i) * (uint32_t)T + (uint32_t)k4);
      const i32x4 o{(int)(v.x & 0xffffu), (int)(v.x >> 16), (int)(v.y & 0xffffu), (int)(v.y >> 16)};
      __builtin_nontemporal_store(o, reinterpret_cast<i32x4 *>(dst));
    }
  }
  __builtin_amdgcn_wave_barrier();
}

// id_pass2 for 8-bit slots: line r's staged rows take 256 bytes from byte
// 256 r, row i of line r rotated by r quads (the 16 writers of one
// instruction touch distinct banks).
template <int QX>
__device__ __forceinline__ void id_pass2(int32_t *leaf_ids, int64_t n_rows, int T, const IdOut &io, const IdPack8 &ids,
                                         int rho0, int te0, int c0, int rho1, int te1, int c1, int lo) {
  // the usual case, uniform over the wave: every row of the wave exists and
  // both lines lie inside the trees [lo, T), so no lane needs a bound check
  if (io.r0w + 64 <= n_rows && te0 - 31 >= lo && te1 + 1 <= T) {
    constexpr int kD = 2 * QX + 1;
    const uint32_t k4 = io.k4;
    const bool w0 = k4 == 4u * (uint32_t)rho0, w1 = k4 == 4u * (uint32_t)rho1;
    if (w0 || w1) {
      unsigned char *dst = reinterpret_cast<unsigned char *>(io.stage) + (w1 ? 256u : 0u) + io.i32;
      u32x4 q0 = ids.q[0], q1 = ids.q[1];
      if (kD >> 2) q1[kD & 3] = w1 ? ids.pend : q1[kD & 3];
      else q0[kD & 3] = w1 ? ids.pend : q0[kD & 3];
      // line 1's rows rotated by one quad: the 16 writers touch distinct banks
      *reinterpret_cast<u32x4 *>(dst + (w1 ? 16u : 0u)) = q0;
      *reinterpret_cast<u32x4 *>(dst + (w1 ? 0u : 16u)) = q1;
    }
    __builtin_amdgcn_wave_barrier();
    const uint32_t b = io.id_base;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int c = r ? c1 : c0;
      const uint32_t v = *reinterpret_cast<const uint32_t *>(reinterpret_cast<const unsigned char *>(io.stage) +
                                                             256 * r + io.i32 + ((k4 + (uint32_t)(c + 16 * r)) & 31u));
      const int64_t row0 = io.r0w + (r ? rho1 : rho0);
      const int tb = (r ? te1 : te0) - 31;
      unsigned char *line = reinterpret_cast<unsigned char *>(leaf_ids + (row0 * T + tb));
      const i32x4 o{(int)(b + (v & 0xffu)), (int)(b + ((v >> 8) & 0xffu)), (int)(b + ((v >> 16) & 0xffu)),
                    (int)(b + (v >> 24))};
      __builtin_nontemporal_store(o, reinterpret_cast<i32x4 *>(line + io.goff));
    }
    __builtin_amdgcn_wave_barrier();
    return;
  }
  const int lane = lane_fresh();
  const int k = lane & 7, i = lane >> 3;
  constexpr int kD = 2 * QX + 1;  // the dword trees 4..7 of chunk QX take
  if (k == rho0 || k == rho1) {
    const int r = k == rho1 ? 1 : 0;
    u32x4 *dst = io.stage + 16 * r + 2 * i;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      u32x4 q = ids.q[j];
      if (j == (kD >> 2)) q[kD & 3] = r ? ids.pend : q[kD & 3];
      dst[(j + r) & 1] = q;
    }
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int c = r ? c1 : c0;
    const uint32_t v = *reinterpret_cast<const uint32_t *>(reinterpret_cast<const unsigned char *>(io.stage) +
                                                           256 * r + 32 * i + ((c + 4 * k + 16 * r) & 31));
    const int64_t row0 = io.r0w + (r ? rho1 : rho0);
    const int rem = (int)min(n_rows - row0, (int64_t)64);
    const int tb = (r ? te1 : te0) - 31;
    const int k4 = 4 * k;
    if (8 * i < rem && k4 >= lo - tb && k4 < T - tb) {
      int32_t *dst = leaf_ids + (row0 * T + tb) + ((uint32_t)(8 * i) * (uint32_t)T + (uint32_t)k4);
      const uint32_t b = io.id_base;
      const i32x4 o{(int)(b + (v & 0xffu)), (int)(b + ((v >> 8) & 0xffu)), (int)(b + ((v >> 16) & 0xffu)),
                    (int)(b + (v >> 24))};
      __builtin_nontemporal_store(o, reinterpret_cast<i32x4 *>(dst));
    }
  }
  __builtin_amdgcn_wave_barrier();
}

// Rows not 16-byte aligned: one int32 per store, a 32-tree group at a time.
__device__ __forceinline__ void flush_scalar(int32_t *leaf_ids, int64_t n_rows, int T, const IdPack8 &ids,
                                             const IdOut &io, int t0) {
  const int ntrees = min(kFastIdGroup, T - t0);
  const int64_t row = io.r0w + (threadIdx.x & 63);
  if (row < n_rows) {
#pragma unroll
    for (int g = 0; g < kFastIdGroup; ++g)
      if (g < ntrees)
        leaf_ids[row * T + t0 + g] = (int)(io.id_base + ((ids.q[g >> 4][(g >> 2) & 3] >> (8 * (g & 3))) & 0xffu));
  }
}
__device__ __forceinline__ void flush_scalar(int32_t *leaf_ids, int64_t n_rows, int T, const IdPack &ids,
                                             const IdOut &io, int t0) {
  const int64_t r0w = io.r0w;
  const int ntrees = min(kFastIdGroup, T - t0);
  const int64_t row = r0w + (threadIdx.x & 63);
  if (row < n_rows) {
#pragma unroll
    for (int g = 0; g < kFastIdGroup; ++g)
      if (g < ntrees) leaf_ids[row * T + t0 + g] = (int)((ids[g >> 3][(g >> 1) & 3] >> (16 * (g & 1))) & 0xffffu);
  }
}

typedef __attribute__((address_space(3))) const float lds_f32;

// LDS byte address of a TT node's feature in this lane's column of the tile:
// xlane + (w & 0xffff) * ROWS * 4 in one v_mad_u32_u16, which multiplies the
// low 16 bits of the record word (the feature) as they are, so the child
// offset in the high half needs no mask.
template <int ROWS>
__device__ __forceinline__ uint32_t tt_xaddr(uint32_t w, uint32_t xlane) {
  static_assert(ROWS * 4 < 65536, "the row stride must fit the 16-bit multiplier");
  uint32_t r;
  asm("v_mad_u32_u16 %0, %1, %2, %3" : "=v"(r) : "v"(w), "s"((uint32_t)ROWS * 4u), "v"(xlane));
  return r;
}

// The values of tree t's leaf reached with walk state s (byte offset of
// the record: PTT heap index 2^LG + slot, TT node index), vector leaves.
template <int MODE, int LG>
__device__ __forceinline__ const float *fast_vec_leaf(const FastArgs &a, int t, uint32_t s) {
  const uint32_t idx = MODE == 0 ? (s >> 3) - (1u << LG) : ((s >> 3) & ((1u << LG) - 1u));
  // (clamped to the table's row so that even a malformed table cannot read outside it)
  return a.vec + ((size_t)min(t, a.out.T - 1) * a.vec_stride + min(idx, (uint32_t)a.vec_stride - 1u)) * a.LD;
}

// Leaf ids and sums of one chunk's trees tb .. tb + TC - 1 (chunk index QP
// within its 32-tree group) from their leaf records: each id into its slot,
// the lines that end inside the chunk out, the values into the sums.
template <int MODE, int LG, int KM, int ROWS, int BUDGET, int QP>
__device__ __forceinline__ void fast_leaves(const FastArgs &a, const uint2 (&lrs)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::TC],
                                            int tb, double (&acc)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::KMAX],
                                            typename FastCfg<MODE, LG, KM, ROWS, BUDGET>::Pack &ids, int cls,
                                            const IdOut &io) {
  using C = FastCfg<MODE, LG, KM, ROWS, BUDGET>;
  constexpr int TC = C::TC;
#pragma unroll
  for (int g = 0; g < TC; ++g) {
    const int t = tb + g;
    const uint2 lr = lrs[g];
    if (C::DEFER && g >= 4 && io.on) {  // held until the lines that end at tree tb + 3 have left
      hold_id(ids, g, lr.y);
    } else {
      put_id(ids, QP * TC + g, lr.y);
    }
    if (!C::DEFER && ((QP * TC + g) & 3) == 3 && g < TC - 1 && io.on) {  // lines that end at tree t, within the chunk
      const int c = (QP * TC + g + 1) & 31;
      uint32_t m = (uint32_t)(a.id_phase >> (8 * (c >> 2))) & 0xffu;
      while (m) {
        const int rho = __builtin_ctz(m);
        m &= m - 1;
        id_pass(a.leaf_ids, a.n_rows, a.out.T, io, ids, rho, t, c, io.t_begin);
      }
    }
    if (t < a.out.T && !C::GV) {  // (GV: the values are added by the caller)
      const double v = (double)as_float(lr.x);
      if (C::MULTI && a.vec) {
        // vector leaves are added by the caller
      } else if (C::MULTI) {
        // the column is uniform across the wave: one register-indexed update
        const int k = __builtin_amdgcn_readlane(cls, g) & (C::KMAX - 1);
        acc[k] += v;
      } else {
        acc[0] += v;
      }
    }
  }
  // rows not 16-byte aligned: a 32-tree group's ids leave at once, by scalar
  // stores (here with LAG, whose groups end one chunk late; else after the group)
  if (C::LAG && QP == C::CPF - 1 && a.leaf_ids && !a.ids_vec)
    flush_scalar(a.leaf_ids, a.n_rows, a.out.T, ids, io, tb - (C::CPF - 1) * TC);
}

// Chunks of 8 trees (DEFER): the lines that ended at tree tb + 3 of the
// chunk with index QX in its group (first tree tb) leave, then the ids of
// the chunk's last four trees take their slots.
template <int QX, class P>
__device__ __forceinline__ void fast_deferred(const FastArgs &a, P &ids, int tb, const IdOut &io) {
  constexpr int kC = (QX * 8 + 4) & 31;  // slot of tree tb + 3 - 31
  uint32_t m = (uint32_t)(a.id_phase >> (8 * (kC >> 2))) & 0xffu;
  while (m) {
    const int rho = __builtin_ctz(m);
    m &= m - 1;
    id_pass(a.leaf_ids, a.n_rows, a.out.T, io, ids, rho, tb + 3, kC, io.t_begin);
  }
  put_pending<QX>(ids);
}

template <int MODE, int LG, int KM, int ROWS, int BUDGET, int B, int Q>
__device__ __forceinline__ void fast_chunk(const FastArgs &a, int c, uint4 (*tbuf)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::CHUNK16],
                                           const float *xs, uint32_t lane4,
                                           double (&acc)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::KMAX],
                                           typename FastCfg<MODE, LG, KM, ROWS, BUDGET>::Pack &ids, int &cls, int &dep,
                                           float2 (&vh)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::VH],
                                           uint2 (&lh)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::LH],
                                           float (&gv)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::GVH],
                                           int (&gk)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::GKH], const IdOut &io) {
  using C = FastCfg<MODE, LG, KM, ROWS, BUDGET>;
  constexpr int TC = C::TC;
  constexpr int TB = C::TB;
  // chunk c is in tbuf[B] (the barrier that ended the previous chunk made it
  // visible); fetch chunk c+1 into registers while walking chunk c
  const bool more = c + 1 < a.n_chunks;
  // The chunk's root records (PTT: heap index 1, at byte 8 of a block; TT:
  // node 0) are the same for every lane. In 1024-row workgroups they come
  // by scalar loads (issued here, used after the chunk's leaf-id passes) and
  // the walk's first level reads no node record from LDS: one LDS read of
  // the 16 of a depth-8 walk, about 3% of the headline's time. With fewer
  // waves per CU the scalar loads' wait at each chunk costs more than that
  // (measured on the 512-row 7-class and 256-row leaf-wise shapes), and the
  // root comes from LDS like the other levels.
  constexpr bool kRootS = ROWS >= 1024;
  constexpr uint32_t kRootOff = (MODE == 0 || MODE == 3) ? 8u : 0u;
  typedef __attribute__((address_space(4))) const uint32_t cword_t;
  uint32_t root_t[kRootS ? TC : 1], root_f[kRootS ? TC : 1];
  if constexpr (kRootS) {
    const cword_t *cb = (const cword_t *)(reinterpret_cast<const unsigned char *>(a.blocks) + (size_t)c * TC * TB);
#pragma unroll
    for (int g = 0; g < TC; ++g) {
      root_t[g] = cb[(g * TB + kRootOff) / 4];
      root_f[g] = cb[(g * TB + kRootOff) / 4 + 1];
    }
  }
  // TT: lane g holds the depth of tree g of the chunk, loaded one chunk ahead
  // and before the blocks (waiting for a load issued behind the prefetch
  // would mean waiting for the whole prefetch)
  int dep_next = 0;
  if (MODE == 1 || MODE == 2) dep_next = a.tree_depth[min((more ? c + 1 : c) * TC + ((int)threadIdx.x & (TC - 1)), a.out.T - 1)];
  __builtin_amdgcn_sched_barrier(0);
  ChunkPrefetch<ROWS, C::CHUNK16> next;
  next.load(a.blocks + (size_t)(more ? c + 1 : c) * C::CHUNK16);
  // multi-output: lane g of every wave holds the output column of tree g of
  // the chunk (loaded one chunk ahead, like the blocks)
  int cls_next = 0;
  if (C::MULTI && !a.vec)
    cls_next = a.tree_class[min((more ? c + 1 : c) * TC + ((int)threadIdx.x & (TC - 1)), a.out.T - 1)];
  const int t0 = c * TC;
  // the lines that ended with the previous chunk (with LAG: the one before,
  // whose ids were taken after this chunk's predecessor's walk) leave now,
  // behind the prefetch: a wait for the prefetch then never waits for their
  // stores
  constexpr int kLag = C::LAG ? 1 : 0;
  constexpr int kQE = (Q + C::CPF - kLag) % C::CPF;  // the chunk that ended, within its group
  const bool ended = io.on && t0 - kLag * TC > io.t_begin;
  if (ended) {
    constexpr int kC = (kQE * TC) & 31;
    const uint32_t m_end = ((kQE * TC) & 3) == 0 ? (uint32_t)(a.id_phase >> (8 * (kC >> 2))) & 0xffu : 0u;
    if constexpr (C::DEFER) {
      // the lines that ended inside that chunk, then its last ids, then the
      // lines that ended with it: one staging for both when each of the two
      // trees ends the lines of a single residue (tree counts of 4 mod 8)
      constexpr int kQX = (Q + 2 * C::CPF - 1 - kLag) % C::CPF;
      constexpr int kCI = (kQX * 8 + 4) & 31;
      const uint32_t m_in = (uint32_t)(a.id_phase >> (8 * (kCI >> 2))) & 0xffu;
      const int tb = t0 - (1 + kLag) * TC;  // first tree of the chunk that ended
      if (__builtin_popcount(m_in) == 1 && __builtin_popcount(m_end) == 1) {
        id_pass2<kQX>(a.leaf_ids, a.n_rows, a.out.T, io, ids, __builtin_ctz(m_in), tb + 3, kCI, __builtin_ctz(m_end),
                      tb + TC - 1, kC, io.t_begin);
        put_pending<kQX>(ids);
      } else {
        fast_deferred<kQX>(a, ids, tb, io);
        for (uint32_t m = m_end; m; m &= m - 1)
          id_pass(a.leaf_ids, a.n_rows, a.out.T, io, ids, __builtin_ctz(m), t0 - kLag * TC - 1, kC, io.t_begin);
      }
    } else {
      for (uint32_t m = m_end; m; m &= m - 1)
        id_pass(a.leaf_ids, a.n_rows, a.out.T, io, ids, __builtin_ctz(m), t0 - kLag * TC - 1, kC, io.t_begin);
    }
  }
  __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the walk
  const unsigned char *base = reinterpret_cast<const unsigned char *>(tbuf[B]);
  const unsigned char *xb = reinterpret_cast<const unsigned char *>(xs);
  uint32_t s[TC];
  if (MODE == 0 || MODE == 3) {
    // Software-pipelined in issue order: LDS reads complete in order, so the
    // node reads of all TC trees go first, then their feature reads, then
    // each tree's step immediately issues its next node read; every wait is
    // for the oldest read and about TC reads stay in flight per wave.
    uint2 rec[TC];
    float xv[TC];
    if constexpr (kRootS) {
      // level 0 from the scalar root records: heap index 1 -> 2 or 3
#pragma unroll
      for (int g = 0; g < TC; ++g)
        xv[g] = *reinterpret_cast<const float *>(xb + root_f[g] * (ROWS * 4u) + lane4);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < TC; ++g) {
        s[g] = xv[g] < as_float(root_t[g]) ? 16u : 24u;
        if (LG > 1) rec[g] = *reinterpret_cast<const uint2 *>(base + g * TB + s[g]);
      }
    } else {
#pragma unroll
      for (int g = 0; g < TC; ++g) {
        s[g] = 8u;  // heap index 1
        rec[g] = *reinterpret_cast<const uint2 *>(base + g * TB + 8u);
      }
    }
#pragma unroll
    for (int lvl = kRootS ? 1 : 0; lvl < LG; ++lvl) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < TC; ++g)
        xv[g] = *reinterpret_cast<const float *>(xb + __umul24(rec[g].y, ROWS * 4u) + lane4);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < TC; ++g) {
        s[g] = 2u * s[g] + (xv[g] < as_float(rec[g].x) ? 0u : 8u);  // Algorithm 3's heap step, in bytes
        if (lvl + 1 < LG) rec[g] = *reinterpret_cast<const uint2 *>(base + g * TB + s[g]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  } else {
    int levels = 0;
#pragma unroll
    for (int g = 0; g < TC; ++g) levels = max(levels, __builtin_amdgcn_readlane(dep, g));
    // Pipelined like the PTT walk: all feature reads of a level are issued
    // before the first is used, and each tree's next node read right after
    // its step (the read after the last level is unused but in bounds: every
    // record's children lie in its own tree).
    const uint32_t xlane = (uint32_t)(uintptr_t)xs + lane4;
    uint64_t rec[TC];  // {threshold bits, feature | 8 * right << 16}, one 8-byte read
    float xv[TC];
    if constexpr (kRootS) {
      // level 0 from the scalar root records (a chunk of leaves only, levels
      // 0, takes the step too: a leaf loops to itself)
#pragma unroll
      for (int g = 0; g < TC; ++g)
        xv[g] = *reinterpret_cast<lds_f32 *>((uintptr_t)(xlane + (root_f[g] & 0xffffu) * (ROWS * 4u)));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < TC; ++g) {
        s[g] = (root_f[g] >> 16) - (xv[g] < as_float(root_t[g]) ? 8u : 0u);
        rec[g] = *reinterpret_cast<const uint64_t *>(base + g * TB + s[g]);
      }
    } else {
#pragma unroll
      for (int g = 0; g < TC; ++g) {
        s[g] = 0u;  // root record
        rec[g] = *reinterpret_cast<const uint64_t *>(base + g * TB);
      }
    }
    for (int lvl = kRootS ? 1 : 0; lvl < levels; ++lvl) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < TC; ++g)
        xv[g] = *reinterpret_cast<lds_f32 *>((uintptr_t)tt_xaddr<ROWS>((uint32_t)(rec[g] >> 32), xlane));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < TC; ++g) {
        // Algorithm 2's step: left or right child
        s[g] = (uint32_t)(rec[g] >> 48) - (xv[g] < as_float((uint32_t)rec[g]) ? 8u : 0u);
        rec[g] = *reinterpret_cast<const uint64_t *>(base + g * TB + s[g]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  // PTT: leaf record at the heap index; TT mode 1: after the node records;
  // TT mode 2: from global memory (the index is masked to the tree's 2^LG
  // records, so even a malformed table cannot read outside them). All are
  // read before the first leaf-id store: a load issued behind a store would
  // also wait for the store to complete.
  uint2 lrs[TC];
  if (C::GV) {
    // the leaf slots are the ids; the previous chunk's values (read a walk
    // ago) are added in tree order, then this chunk's are read
#pragma unroll
    for (int g = 0; g < TC; ++g) {
      const uint32_t slot = (s[g] >> 3) & ((1u << LG) - 1u);
      lrs[g] = make_uint2(0u, slot);
      if constexpr (C::MULTI) {
        // the column is uniform across the wave: one register-indexed update
        acc[gk[g]] += (double)gv[g];
        gk[g] = __builtin_amdgcn_readlane(cls, g) & (C::KMAX - 1);
      } else {
        acc[0] += (double)gv[g < C::GVH ? g : 0];
      }
      gv[g < C::GVH ? g : 0] = a.leafv[((size_t)(t0 + g) << LG) | slot];
    }
  }
#pragma unroll
  for (int g = 0; g < TC && !C::GV; ++g) {
    if (MODE == 2)
      lrs[g] = a.leaf[(size_t)(t0 + g) * (1u << LG) + ((s[g] >> 3) & ((1u << LG) - 1u))];
    else
      lrs[g] = *reinterpret_cast<const uint2 *>(base + g * TB + (MODE == 0 ? 0u : (1u << LG) * 8u) + s[g]);
  }
  // vector leaves, two values (VHOLD): the previous chunk's leaves, read
  // a whole walk ago, are added now and this chunk's are read, before the
  // first leaf-id store (a load issued behind a store would also wait for
  // the store), to be added after the next walk
  if (C::VHOLD && a.vec) {
#pragma unroll
    for (int g = 0; g < C::VH; ++g) {
      acc[0] += (double)vh[g].x;
      acc[1] += (double)vh[g].y;
      vh[g] = t0 + g < a.out.T ? *reinterpret_cast<const float2 *>(fast_vec_leaf<MODE, LG>(a, t0 + g, s[g]))
                               : make_float2(0.0f, 0.0f);
    }
  } else if (C::MULTI && a.vec) {
    // longer vectors: every value of every tree's leaf is added here, before
    // the first leaf-id store
#pragma unroll
    for (int g = 0; g < TC; ++g) {
      if (t0 + g < a.out.T) {
        const float *vp = fast_vec_leaf<MODE, LG>(a, t0 + g, s[g]);
#pragma unroll
        for (int k = 0; k < C::KMAX; ++k)
          if (k < a.LD) acc[k] += (double)vp[k];
      }
    }
  }
  if (C::LAG) {
    // the previous chunk's records (read a walk ago), then hold this chunk's
    uint2 prev[TC];
#pragma unroll
    for (int g = 0; g < TC; ++g) {
      prev[g] = lh[g < C::LH ? g : 0];
      lh[g < C::LH ? g : 0] = lrs[g];
    }
    if (t0 > io.t_begin) fast_leaves<MODE, LG, KM, ROWS, BUDGET, (Q + C::CPF - 1) % C::CPF>(a, prev, t0 - TC, acc, ids, cls, io);
  } else {
    fast_leaves<MODE, LG, KM, ROWS, BUDGET, Q>(a, lrs, t0, acc, ids, cls, io);
  }
  cls = cls_next;
  dep = dep_next;
  if (C::BUFS == 2) {
    if (more) next.store(tbuf[B ^ 1]);  // nobody reads tbuf[B^1] during chunk c
    lds_barrier();
  } else {
    lds_barrier();  // every wave is done with the single buffer
    if (more) next.store(tbuf[0]);
    lds_barrier();
  }
}

// The CPF chunks between two leaf-id flushes, unrolled so that buffer
// indices and id slots are compile-time constants.
template <int MODE, int LG, int KM, int ROWS, int BUDGET, int Q>
__device__ __forceinline__ void fast_group(const FastArgs &a, int c0, uint4 (*tbuf)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::CHUNK16],
                                           const float *xs, uint32_t lane4,
                                           double (&acc)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::KMAX],
                                           typename FastCfg<MODE, LG, KM, ROWS, BUDGET>::Pack &ids, int &cls, int &dep,
                                           float2 (&vh)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::VH],
                                           uint2 (&lh)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::LH],
                                           float (&gv)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::GVH],
                                           int (&gk)[FastCfg<MODE, LG, KM, ROWS, BUDGET>::GKH], const IdOut &io) {
  using C = FastCfg<MODE, LG, KM, ROWS, BUDGET>;
  if constexpr (Q < C::CPF) {
    fast_chunk<MODE, LG, KM, ROWS, BUDGET, C::BUFS == 2 ? (Q & 1) : 0, Q>(a, c0 + Q, tbuf, xs, lane4, acc, ids,
                                                                           cls, dep, vh, lh, gv, gk, io);
    fast_group<MODE, LG, KM, ROWS, BUDGET, Q + 1>(a, c0, tbuf, xs, lane4, acc, ids, cls, dep, vh, lh, gv, gk, io);
  }
}

template <int MODE, int LG, int KM, int ROWS, int BUDGET>
__global__ __launch_bounds__(ROWS) void fast_kernel(FastArgs a) {
  using C = FastCfg<MODE, LG, KM, ROWS, BUDGET>;
  constexpr int G = kFastIdGroup;
  // this workgroup's chunks (all of them unless the trees are split)
  const int c_begin = a.split ? (int)blockIdx.y * a.split : 0;
  if (a.split) a.n_chunks = min(c_begin + a.split, a.n_chunks);
  __shared__ __align__(16) uint4 tbuf[C::BUFS][C::CHUNK16];
  __shared__ __align__(16) u32x4 idstage[ROWS / 64][2 * 8 * kIdQuads];
  extern __shared__ __align__(16) float fxs[];  // [F][ROWS]
  const int tid = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * ROWS;
  const int64_t row = r0 + tid;
  const bool valid = row < a.n_rows;
  {
    ChunkPrefetch<ROWS, C::CHUNK16> first;
    first.load(a.blocks + (size_t)c_begin * C::CHUNK16);
    first.store(tbuf[0]);
  }
  {  // each lane copies its own row into column tid of the tile (and only
     // ever reads that column back, so the tile needs no barrier)
    const float *src = a.X + (valid ? row : r0) * a.Fs;
    if (!a.cols && (a.F & 3) == 0 && (reinterpret_cast<uintptr_t>(a.X) & 15) == 0) {
      for (int f = 0; f < a.F; f += 4) {
        const float4 v = valid ? *reinterpret_cast<const float4 *>(src + f) : make_float4(0, 0, 0, 0);
        fxs[(f + 0) * ROWS + tid] = v.x;
        fxs[(f + 1) * ROWS + tid] = v.y;
        fxs[(f + 2) * ROWS + tid] = v.z;
        fxs[(f + 3) * ROWS + tid] = v.w;
      }
    } else {
      for (int f = 0; f < a.F; ++f) fxs[f * ROWS + tid] = valid ? xval(src, a.cols, f) : 0.0f;
    }
  }
  lds_barrier();
  const uint32_t lane4 = (uint32_t)tid * 4u;
  double acc[C::KMAX];
#pragma unroll
  for (int k = 0; k < C::KMAX; ++k) acc[k] = 0.0;
  typename C::Pack ids;
  int cls = C::MULTI && !a.vec ? a.tree_class[min(c_begin * C::TC + (tid & (C::TC - 1)), a.out.T - 1)] : 0;
  int dep = (MODE == 1 || MODE == 2) ? a.tree_depth[min(c_begin * C::TC + (tid & (C::TC - 1)), a.out.T - 1)] : 0;
  float2 vh[C::VH];
#pragma unroll
  for (int g = 0; g < C::VH; ++g) vh[g] = make_float2(0.0f, 0.0f);
  uint2 lh[C::LH];
#pragma unroll
  for (int g = 0; g < C::LH; ++g) lh[g] = make_uint2(0u, 0u);
  float gv[C::GVH];
#pragma unroll
  for (int g = 0; g < C::GVH; ++g) gv[g] = 0.0f;
  int gk[C::GKH];
#pragma unroll
  for (int g = 0; g < C::GKH; ++g) gk[g] = 0;
  const IdOut io = make_id_out<ROWS>(a.leaf_ids != nullptr && a.ids_vec != 0, idstage[tid >> 6], c_begin * C::TC,
                                     (uint32_t)a.id_base, a.out.T);
  for (int c = c_begin; c < a.n_chunks; c += C::CPF) {  // chunk counts are multiples of CPF
    fast_group<MODE, LG, KM, ROWS, BUDGET, 0>(a, c, tbuf, fxs, lane4, acc, ids, cls, dep, vh, lh, gv, gk, io);
    if (!C::LAG && a.leaf_ids && !a.ids_vec) flush_scalar(a.leaf_ids, a.n_rows, a.out.T, ids, io, c * C::TC);
  }
  if constexpr (C::DEFER && !C::LAG)  // the last chunk's inside lines and ids
    if (io.on) fast_deferred<C::CPF - 1>(a, ids, a.n_chunks * C::TC - C::TC, io);
  if (C::LAG) {
    // the lines that ended with the next-to-last chunk, then the last
    // chunk's leaf ids and sums
    const int t_last = a.n_chunks * C::TC - C::TC;  // first tree of the last chunk
    if constexpr (C::DEFER)
      if (io.on && t_last - C::TC >= io.t_begin) fast_deferred<(2 * C::CPF - 2) % C::CPF>(a, ids, t_last - C::TC, io);
    constexpr int kC = ((C::CPF - 1) * C::TC) & 31;
    if ((kC & 3) == 0 && io.on && t_last > io.t_begin) {
      uint32_t m = (uint32_t)(a.id_phase >> (8 * (kC >> 2))) & 0xffu;
      while (m) {
        const int rho = __builtin_ctz(m);
        m &= m - 1;
        id_pass(a.leaf_ids, a.n_rows, a.out.T, io, ids, rho, t_last - 1, kC, io.t_begin);
      }
    }
    uint2 last[C::TC];
#pragma unroll
    for (int g = 0; g < C::TC; ++g) last[g] = lh[g < C::LH ? g : 0];
    fast_leaves<MODE, LG, KM, ROWS, BUDGET, C::CPF - 1>(a, last, t_last, acc, ids, cls, io);
    if constexpr (C::DEFER)
      if (io.on) fast_deferred<C::CPF - 1>(a, ids, t_last, io);
  }
  if (C::GV) {  // the last chunk's values
#pragma unroll
    for (int g = 0; g < C::GVH; ++g) {
      if constexpr (C::MULTI)
        acc[gk[g]] += (double)gv[g];
      else
        acc[0] += (double)gv[g];
    }
  }
  if (C::VHOLD && a.vec) {  // the last chunk's 2-vector leaves
#pragma unroll
    for (int g = 0; g < C::VH; ++g) {
      acc[0] += (double)vh[g].x;
      acc[1] += (double)vh[g].y;
    }
  }
  if (io.on) {
    // the rest of every row's last line: from its start (tree t_pad - 32 + 4k)
    // to the end (k = 0: the lines that ended with the last chunk)
    const int t_pad = a.n_chunks * C::TC;
    for (int k = 0; k < 8; ++k) {
      uint32_t m = (uint32_t)(a.id_phase >> (8 * k)) & 0xffu;
      while (m) {
        const int rho = __builtin_ctz(m);
        m &= m - 1;
        id_pass(a.leaf_ids, a.n_rows, a.out.T, io, ids, rho, t_pad - 1, 0, max(io.t_begin, t_pad - 32 + 4 * k));
      }
    }
  }
  if (valid) {
    if (a.split) {
      double *dst = a.partial + ((size_t)blockIdx.y * a.n_rows + row) * a.out.K;
#pragma unroll
      for (int k = 0; k < C::KMAX; ++k)
        if (k < a.out.K) dst[k] = acc[k];
    } else {
      finish_row<C::KMAX>(a.out, acc, row);
    }
  }
}


template <int MODE, int KM, int ROWS, int BUDGET, int LG = 1>
FastFn pick_fast(int lg) {
  if constexpr (LG > kFastMaxLgFor<MODE>) {
    return nullptr;
  } else {
    if (lg == LG) return fast_kernel<MODE, LG, KM, ROWS, BUDGET>;
    return pick_fast<MODE, KM, ROWS, BUDGET, LG + 1>(lg);
  }
}

}  // namespace
}  // namespace hb
