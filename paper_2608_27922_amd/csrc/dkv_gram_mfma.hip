// Key-key Gram stages of the DensityKV update on bf16 MFMA (gfx950).
//
// Every Gram stage evaluates Soft-Riesz weights w(k_i, k_j) (Eq. 2) for a set
// of "row" items against a stream of "column" items and reduces them per row:
//
//   k_score_mfma       rows = candidates, columns = bank states:
//                      S_x = sum_i RNE(w_ix bs_i), Wcol_x = sum_i W_ix  (Eq. 6)
//   k_first_part_mfma  per bank state, over the first 256 ordered candidates:
//                      64-candidate chunk sums (the prefix checkpoints of
//                      Eqs. 8-9) and the first prefix that reaches tau b
//   k_chunk_part_mfma  the chunk sums of the rest of the order, and
//   k_cross_mfma       the whole crossing search, for the groups that the first
//                      part leaves open (k_cross_plan, Eqs. 9-11)
//   k_rowsum_mfma      row sums: the r* fix-up, the exact maintenance (Supp. C)
//                      and the from-scratch bank density (Eq. 3)
//
// The column range of every Gram is split over workgroups (grid dimension y);
// partial integer sums are combined with 64-bit atomic adds, which are exact
// and order-independent.
//
// Layout: a workgroup of 4 waves owns 128 row items; wave w owns 32 of them,
// held for the whole kernel as the B operand of v_mfma_f32_32x32x16_bf16
// (lane l <-> row item l % 32).  Column items stream through LDS in stages of 64
// (three stages resident, loaded global -> LDS directly, key rows swizzled)
// and form the A operand, so each lane ends up with 16 weights of its own row
// item and reduces them in registers.
//
// Exactness: with keys on the 1/64 grid every partial sum of the contraction
// is an exact multiple of 2^-18 below 2^24 units, so the MFMA result
//   u = (|k_i|^2 + |k_j|^2 - 2 <k_i, k_j>) / sigma^2
// is exact.  The norms enter through one extra K step (each norm / sigma^2 is
// split exactly into three bf16 pieces) and the row keys are pre-scaled by
// -2 / sigma^2 (exact in bf16).  The epilogue is the binary32 contract:
// t = 1 + u, t^p, correctly rounded reciprocal (rcp + one FMA correction, exact
// for every significand), RNE(w * 2^23) via one FMA, integer sums.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "dkv_internal.hpp"

namespace dkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;  // waves per workgroup of the crossing search, and of the Gram stages at D <= 128
// Waves per workgroup of the Gram stages: 8 at descriptor dimension 256, whose
// three column stages (about 100 KB of LDS) allow one workgroup per CU, so that
// each SIMD still holds two waves.
template <int D>
constexpr int gram_waves() { return D > 128 ? 8 : kWaves; }
constexpr int kCT = 32;  // column items per MFMA tile
constexpr int kSI = 64;  // column items per LDS stage (two tiles, two independent MFMA chains)

template <int D>
struct TileCfg {
  static constexpr int kSteps = D / 16;     // K steps over the key
  static constexpr int kChunks = D / 8;     // 16-byte chunks per key
};

__device__ __forceinline__ uint16_t bf16_rne_bits(float f) { return f32_to_bf16_bits(f); }

// Exact split of x (at most 24 significant bits) into three bf16 values.
__device__ __forceinline__ void split3(float x, uint16_t &h, uint16_t &m, uint16_t &l) {
  h = bf16_rne_bits(x);
  float r = x - bf16_bits_to_f32(h);
  m = bf16_rne_bits(r);
  float r2 = r - bf16_bits_to_f32(m);
  l = bf16_rne_bits(r2);
}

constexpr uint16_t kOne = 0x3F80;  // bf16 1.0

// FOLD: the MFMA already added the 1 of t = 1 + u (exact when sigma^2 <= 2^11,
// where every partial sum stays below 2^24 units of 2^-12 / sigma^2).
template <int P, bool FOLD>
__device__ __forceinline__ uint32_t weight_raw(float u, float scale) {
  // raw bits of fma(w, scale, 2^23): kMagic + RNE(w * scale)
  const float t = FOLD ? u : 1.0f + u;
  float tp = t;
  if constexpr (P >= 2) tp = t * t;
  if constexpr (P == 4) tp = tp * tp;
  const float w = clamp_weight(rcp_rn(tp));
  return __float_as_uint(__builtin_fmaf(w, scale, 8388608.0f));
}

// Source of retention descriptors of dimension D: row r's descriptor is k[r]
// (rows of D elements) or, for the [K; V] geometry (SPLIT), the concatenation
// [k[r]; v[r]] of two rows of D / 2 elements.  desc_chunk gives its 16-byte
// chunk c (8 bf16).
struct Desc {
  const uint16_t *k;
  const uint16_t *v;
};

template <int D, bool SPLIT>
__device__ __forceinline__ const uint16_t *desc_chunk(const Desc &s, int64_t row, int c) {
  if constexpr (!SPLIT) {
    return s.k + row * D + 8 * c;
  } else {
    constexpr int H = D / 2;
    return c < H / 8 ? s.k + row * H + 8 * c : s.v + row * H + 8 * (c - H / 8);
  }
}

// Row fragment: B operand of every K step for this lane's row item.
template <int D>
struct RowFrag {
  bf16x8 b[TileCfg<D>::kSteps + 1];
};

// Load the B operand for row item (lane % 32): keys scaled by -2/sigma^2, then
// the aug step [1, 1, 1, n_hi, n_mid, n_lo, fold, 0] (half 0) / zeros (half 1).
template <int D, bool FOLD, bool SPLIT>
__device__ __forceinline__ void load_row_frag(RowFrag<D> &rf, const Desc &src, int64_t row, float norm, bool valid,
                                              float neg2_inv_s2, float inv_s2) {
  const int h = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int kk = 0; kk < TileCfg<D>::kSteps; ++kk) {
    u32x4 raw = {0, 0, 0, 0};
    if (valid) raw = *reinterpret_cast<const u32x4 *>(desc_chunk<D, SPLIT>(src, row, 2 * kk + h));
    u32x4 sc;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // both halves times a power of two (exact), back to bf16 in one packed conversion
      const float lo = __uint_as_float(raw[q] << 16) * neg2_inv_s2;
      const float hi = __uint_as_float(raw[q] & 0xFFFF0000u) * neg2_inv_s2;
      sc[q] = pack_bf16x2(lo, hi);
    }
    rf.b[kk] = __builtin_bit_cast(bf16x8, sc);
  }
  u32x4 aug = {0, 0, 0, 0};
  if (valid && h == 0) {
    uint16_t nh, nm, nl;
    split3(norm * inv_s2, nh, nm, nl);
    aug[0] = (uint32_t)kOne | ((uint32_t)kOne << 16);
    aug[1] = (uint32_t)kOne | ((uint32_t)nh << 16);
    aug[2] = (uint32_t)nm | ((uint32_t)nl << 16);
    aug[3] = FOLD ? (uint32_t)kOne : 0u;
  }
  rf.b[TileCfg<D>::kSteps] = __builtin_bit_cast(bf16x8, aug);
}

// ---------------------------------------------------------------------------
// Column stages in LDS: 64 column items per stage, three stages resident (two
// loading while one is used).  Keys go global -> LDS with 16-byte direct-to-LDS
// loads (no VGPR staging); a key row is 2 d bytes with its 16-byte chunk c
// stored at c ^ (row % chunks), so that the A-operand reads (32 rows, one chunk
// each) are free of bank conflicts.  Each item's extra K step (column_aug,
// precomputed per update) and, for the score, its score scale follow.
// ---------------------------------------------------------------------------
template <int D, int W = kWaves>
struct SCfg {
  static constexpr int CH = D / 8;             // 16-byte chunks per key row
  static constexpr int RB = 2 * D;             // key row bytes
  static constexpr int RPL = 1024 / RB;        // rows per 1 KB load
  static constexpr int NB = kSI * RB / 1024;   // 1 KB loads per stage
  static constexpr int PER = NB / W;           // key loads per thread per stage
  static constexpr int KEYB = kSI * RB;        // key bytes per stage
  static constexpr int AUGB = kSI * 16;        // aug bytes per stage
  static constexpr int ITEMS = kSI / W;       // aug / scale items per wave (its lanes 0 .. ITEMS - 1)
  static_assert(NB % W == 0 && kSI % W == 0, "loads split evenly over the waves");
};
// direct-to-LDS loads per thread per stage: keys, aug (+ score scale)
template <int D, bool kBs, int W = kWaves>
constexpr int stage_ops() { return SCfg<D, W>::PER + 1 + (kBs ? 1 : 0); }

typedef __attribute__((address_space(3))) void lds_void;

// Global rows fetched by this thread for the stage starting at column j0 (its
// key loads, then its aug / scale item); items past ncols repeat the last one.
template <int D, int W>
using StageRows = int32_t[SCfg<D, W>::PER + 1];

template <int D, int W, class RowOf>
__device__ __forceinline__ void stage_rows(StageRows<D, W> &rows, int j0, int ncols, RowOf row_of) {
  using C = SCfg<D, W>;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
#pragma unroll
  for (int q = 0; q < C::PER; ++q) {
    const int r = (wave * C::PER + q) * C::RPL + l / C::CH;
    rows[q] = (int32_t)row_of(min(j0 + r, ncols - 1));
  }
  rows[C::PER] = (int32_t)row_of(min(j0 + C::ITEMS * wave + l % C::ITEMS, ncols - 1));
}

// Word 3 of a raw buffer resource: 32-bit data format, no swizzle, no
// thread-id addressing.
constexpr int kBufferRsrcWord3 = 0x00020000;

// One 16-byte (4-byte) raw buffer load per lane to LDS, dst + 16 lane
// (dst + 4 lane), from base + voff, with the bytes [base, base + nbytes) as
// the buffer's extent.
__device__ __forceinline__ void buffer_to_lds16(const void *base, int nbytes, int voff, char *dst) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, nbytes, kBufferRsrcWord3);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)dst, 16, voff, 0, 0, 0);
}
__device__ __forceinline__ void buffer_to_lds4(const void *base, int nbytes, int voff, char *dst) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, nbytes, kBufferRsrcWord3);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)dst, 4, voff, 0, 0, 0);
}

// Stage loads.  Every row of a call lies in one bank's region of its arrays,
// rows [row0, row0 + nrows) (uniform), so whole-key-row descriptors go through
// raw buffer loads to LDS over that region: with a global load to LDS in flight
// the compiler counts every later LDS read as possibly out of order and waits
// for all of them before each use.  [K; V] descriptors, whose two halves come
// from two arrays chosen per lane, keep the global loads to LDS.
template <int D, bool kBs, bool SPLIT, int W = kWaves>
__device__ __forceinline__ void stage_dma(const StageRows<D, W> &rows, const Desc &keys,
                                          const uint4 *augs, const float *bs, char *kb, char *ab, float *sb,
                                          int64_t row0, int nrows) {
  using C = SCfg<D, W>;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  if constexpr (!SPLIT) {
    const void *kbase = keys.k + row0 * D;
    const int kbytes = nrows * C::RB;
#pragma unroll
    for (int q = 0; q < C::PER; ++q) {
      const int blk = wave * C::PER + q;
      const int r = blk * C::RPL + l / C::CH;
      const int c = (l % C::CH) ^ (r % C::CH);
      buffer_to_lds16(kbase, kbytes, (int)(rows[q] - row0) * C::RB + 16 * c, kb + blk * 1024);
    }
  } else {
#pragma unroll
    for (int q = 0; q < C::PER; ++q) {
      const int blk = wave * C::PER + q;
      const int r = blk * C::RPL + l / C::CH;
      const int c = (l % C::CH) ^ (r % C::CH);
      __builtin_amdgcn_global_load_lds((void *)desc_chunk<D, SPLIT>(keys, (int64_t)rows[q], c),
                                       (lds_void *)(kb + blk * 1024), 16, 0, 0);
    }
  }
  // items ITEMS w .. ITEMS (w + 1) - 1: lanes 0 .. ITEMS - 1 of wave w (LDS address = base + lane * size)
  if (l < C::ITEMS) {
    const int rel = (int)(rows[C::PER] - row0);
    buffer_to_lds16(augs + row0, nrows * 16, rel * 16, ab + 16 * C::ITEMS * wave);
    if constexpr (kBs) buffer_to_lds4(bs + row0, nrows * 4, rel * 4, reinterpret_cast<char *>(sb + C::ITEMS * wave));
  }
}

// Stages whose rows are consecutive (row i of a stage = the stage's first row
// + i: bank slots in order, or the ordered candidates): each lane's byte
// offsets are the same for every stage, and the stage's first row goes into the
// uniform buffer base, so no per-stage row arithmetic runs on the VALU.
template <int D, int W = kWaves>
struct StageOff {
  int key[SCfg<D, W>::PER];  // key loads: row r of the stage, swizzled chunk c, as r RB + 16 c
  int item;                  // aug / scale item of lanes 0 .. ITEMS - 1 of each wave: ITEMS w + lane
};

template <int D, int W = kWaves>
__device__ __forceinline__ StageOff<D, W> stage_offsets() {
  using C = SCfg<D, W>;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  StageOff<D, W> o;
#pragma unroll
  for (int q = 0; q < C::PER; ++q) {
    const int r = (wave * C::PER + q) * C::RPL + l / C::CH;
    o.key[q] = r * C::RB + 16 * ((l % C::CH) ^ (r % C::CH));
  }
  o.item = C::ITEMS * wave + l % C::ITEMS;
  return o;
}

// Loads of the stage whose first row is row0 + first (whole-row descriptors).
// The buffers end where the region [row0, row0 + nrows) ends, so rows past it
// read as zero; rows past the Gram's last column are real rows of the region,
// masked by the epilogue like the repeated last row they replace.
template <int D, bool kBs, int W = kWaves>
__device__ __forceinline__ void stage_dma_seq(const StageOff<D, W> &o, int first, const uint16_t *keys,
                                              const uint4 *augs, const float *bs, char *kb, char *ab, float *sb,
                                              int64_t row0, int nrows) {
  using C = SCfg<D, W>;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  const int64_t r0 = row0 + first;
  const int left = nrows - first;  // rows from the stage's first to the region's end
#pragma unroll
  for (int q = 0; q < C::PER; ++q)
    buffer_to_lds16(keys + r0 * D, left * C::RB, o.key[q], kb + (wave * C::PER + q) * 1024);
  if (l < C::ITEMS) {
    buffer_to_lds16(augs + r0, left * 16, o.item * 16, ab + 16 * C::ITEMS * wave);
    if constexpr (kBs) buffer_to_lds4(bs + r0, left * 4, o.item * 4, reinterpret_cast<char *>(sb + C::ITEMS * wave));
  }
}

// s_waitcnt immediate (gfx9 encoding): at most n vector-memory operations
// outstanding and no LDS operation outstanding (expcnt left alone).
constexpr int waitcnt_vm_lgkm0(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

// Stage barrier without a memory fence: each thread has waited for its own
// loads of the stage about to be read, so the loads of later stages stay in
// flight; the "memory" clobber keeps LDS accesses from moving across it.
__device__ __forceinline__ void stage_barrier() { asm volatile("s_barrier" ::: "memory"); }

// u for both 32-item tiles of a stage: A fragments from the swizzled key rows
// and the aug step, two interleaved MFMA chains.
template <int D, int AHEAD>
__device__ __forceinline__ void stage_u(const char *kb, const char *ab, const RowFrag<D> &rf, f32x16 &u0,
                                        f32x16 &u1) {
  constexpr int KS = TileCfg<D>::kSteps;
  const int l = threadIdx.x & 63, h = l >> 5, r0 = l & 31, r1 = 32 + r0;
  bf16x8 a0[KS + 1], a1[KS + 1];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    const int c = 2 * kk + h;
    a0[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(
                                            kb + r0 * SCfg<D>::RB + 16 * (c ^ (r0 % SCfg<D>::CH))));
    a1[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(
                                            kb + r1 * SCfg<D>::RB + 16 * (c ^ (r1 % SCfg<D>::CH))));
  }
  // the aug step: both half-waves read the item's 16 bytes; the row fragment's
  // second half is zero, so the h = 1 copy contributes nothing
  a0[KS] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(ab + 16 * r0));
  a1[KS] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(ab + 16 * r1));
  f32x16 x0 = {}, x1 = {};
#pragma unroll
  for (int kk = 0; kk <= KS; ++kk) {
    x0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[kk], rf.b[kk], x0, 0, 0, 0);
    x1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[kk], rf.b[kk], x1, 0, 0, 0);
  }
  // AHEAD > 0: keep AHEAD fragment reads in flight ahead of the MFMAs (the LDS
  // latency is several MFMAs long), i.e. AHEAD reads, then one MFMA and one read
  // at a time; 0 leaves the order to the compiler (kernels with less register room)
  if constexpr (AHEAD > 0) {
    constexpr int kFrags = 2 * (KS + 1), kAhead = kFrags < AHEAD ? kFrags : AHEAD;
    __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);  // LDS reads
#pragma unroll
    for (int i = 0; i < kFrags - kAhead; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAhead, 0);
  }
  u0 = x0;
  u1 = x1;
}

// Tile-granular software pipeline of the Gram stages (descriptors of up to 128
// elements): the 9 MFMAs of the next 32-column tile are issued interleaved with
// the epilogue of the current tile, so that one wave keeps the matrix cores and
// the VALU busy at the same time instead of relying on other waves.
// frag_offsets: byte offsets of this lane's A fragments in a stage buffer
// (tile 0; tile 1 is 32 rows further: rows r and r + 32 share the swizzle).
template <int D>
__device__ __forceinline__ void frag_offsets(int (&off)[TileCfg<D>::kSteps]) {
  static_assert(32 % SCfg<D>::CH == 0, "rows r and r + 32 share the swizzle");
  const int l = threadIdx.x & 63, h = l >> 5, r0 = l & 31;
#pragma unroll
  for (int kk = 0; kk < TileCfg<D>::kSteps; ++kk) off[kk] = r0 * SCfg<D>::RB + 16 * ((2 * kk + h) ^ (r0 % SCfg<D>::CH));
}
// The exact t = 1 + d2 / sigma^2 of one 32-column tile (half 0 or 1 of a
// stage): the column items' A fragments from LDS times the row fragment, one
// MFMA chain
template <int D>
__device__ __forceinline__ f32x16 tile_mfma(const char *kb, const char *ab, int half, const RowFrag<D> &rf,
                                            const int (&off)[TileCfg<D>::kSteps]) {
  constexpr int KS = TileCfg<D>::kSteps;
  const int r0 = threadIdx.x & 31;
  bf16x8 a[KS + 1];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk)
    a[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(kb + 32 * half * SCfg<D>::RB + off[kk]));
  a[KS] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(ab + 16 * (32 * half + r0)));
  f32x16 x = {};
#pragma unroll
  for (int kk = 0; kk <= KS; ++kk) x = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk], rf.b[kk], x, 0, 0, 0);
  return x;
}
// Scheduling of the region that holds one tile_mfma and one tile epilogue:
// LEAD LDS reads first (3 fragments, plus any other reads of the region), then
// per MFMA one read and a slice of the epilogue.
template <int D, int LEAD = 3>
__device__ __forceinline__ void tile_interleave() {
  __builtin_amdgcn_sched_group_barrier(0x100, LEAD, 0);  // LDS reads
#pragma unroll
  for (int i = 0; i <= TileCfg<D>::kSteps; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);  // VALU
  }
}

__device__ __forceinline__ int col_of_reg(int i, int h) { return 8 * (i >> 2) + 4 * h + (i & 3); }

// Sum over this lane's 16 weights (as integers), columns >= nvalid masked out.
template <int P, bool MASK, bool FOLD>
__device__ __forceinline__ uint32_t lane_wsum(const f32x16 &u, int nvalid, int h) {
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    uint32_t raw = weight_raw<P, FOLD>(u[i], 8388608.0f);
    if constexpr (MASK) raw = col_of_reg(i, h) < nvalid ? raw : kMagic;
    s += raw;
  }
  return s - 16u * kMagic;
}

// ---------------------------------------------------------------------------
// Score: rows = candidates, columns = bank states [c0, c1) of this split.
// ---------------------------------------------------------------------------
constexpr int kColsPerSplit = 1024;

template <int D, int P, bool FOLD, bool KV>
__global__ __launch_bounds__(64 * gram_waves<D>(), gram_waves<D>() == 4 ? 3 : 2) void k_score_mfma(dkv_bank bank, const void *seg_k, const void *seg_v,
                                                           Geom g, Prm p, Workspace ws) {
  constexpr int W = gram_waves<D>();
  // One-dimensional grid over (row block, column split, bank), row blocks
  // fastest.  Workgroup L is dispatched to XCD L % 8; ranking the workgroups
  // XCD by XCD (r = workgroups on lower XCDs + L / 8) keeps all the work items
  // of a bank on one XCD, in order, so that its keys and the candidates' stay
  // in that XCD's L2.
  const int nx = (g.N + 32 * W - 1) / (32 * W), ny = (g.Mcap + kColsPerSplit - 1) / kColsPerSplit;
  const int T = (int)gridDim.x, L = (int)blockIdx.x, xcd = L % 8;
  const int r = xcd * (T / 8) + min(xcd, T % 8) + L / 8;
  const int b = r / (nx * ny), by = (r / nx) % ny, bx = r % nx;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const int x = bx * 32 * W + wave * 32 + n;
  const int m = ws.m[b];
  const int c0 = by * kColsPerSplit;
  if (c0 >= m) return;
  const int ncols = min(kColsPerSplit, m - c0);
  constexpr int KB = SCfg<D>::KEYB, AB = SCfg<D>::AUGB;
  __shared__ __attribute__((aligned(1024))) char k0[KB], k1[KB], k2[KB];
  __shared__ __attribute__((aligned(16))) char a0[AB], a1[AB], a2[AB];
  __shared__ __attribute__((aligned(16))) float s0[kSI], s1[kSI], s2[kSI];
  const Desc K{static_cast<const uint16_t *>(seg_k), static_cast<const uint16_t *>(seg_v)};
  const Desc BK{static_cast<const uint16_t *>(bank.k), static_cast<const uint16_t *>(bank.v)};
  const bool rv = x < g.N;
  const size_t xr = (size_t)b * g.N + (rv ? x : 0);
  RowFrag<D> rf;
  load_row_frag<D, FOLD, KV>(rf, K, (int64_t)xr, rv ? ws.cnorm[xr] : 0.0f, rv, -2.0f * p.inv_sigma2, p.inv_sigma2);
  const size_t rb = (size_t)b * g.Mcap + c0;
  const int64_t bank_row0 = (int64_t)b * g.Mcap;  // the stage rows lie in bank b's slots
  auto row_of = [&](int i) -> int64_t { return (int64_t)(rb + i); };
  uint64_t A64 = 0;
  const int ns = (ncols + kSI - 1) / kSI;
  // epilogue of one 32-column tile: integer sum of the scaled score terms
  auto epi = [&](auto mask_tag, const f32x16 &u, const float *tb, int nvalid, uint32_t &sa)
      __attribute__((always_inline)) {
    constexpr bool MASK = decltype(mask_tag)::value;
    float bsv[16];
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const float4 v = *reinterpret_cast<const float4 *>(&tb[8 * gq + 4 * h]);
      bsv[4 * gq + 0] = v.x;
      bsv[4 * gq + 1] = v.y;
      bsv[4 * gq + 2] = v.z;
      bsv[4 * gq + 3] = v.w;
    }
    sa = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float tt = FOLD ? u[i] : 1.0f + u[i];
      float tp = tt;
      if constexpr (P >= 2) tp = tt * tt;
      if constexpr (P == 4) tp = tp * tp;
      const float w = clamp_weight(rcp_rn(tp));
      uint32_t ra = __float_as_uint(__builtin_fmaf(w, bsv[i], 8388608.0f));
      if constexpr (MASK) ra = col_of_reg(i, h) < nvalid ? ra : kMagic;
      sa += ra;
    }
    sa -= 16u * kMagic;
  };
  using Full = std::integral_constant<bool, false>;
  using Part = std::integral_constant<bool, true>;
  constexpr int kOps = stage_ops<D, true, W>();
  StageRows<D, W> rows;
  // stage s: rows s kSI .. of this split; whole-row descriptors take the
  // per-lane offsets of consecutive rows, [K; V] ones (two arrays) the row list
  [[maybe_unused]] const StageOff<D, W> soff = stage_offsets<D, W>();
  auto stage_rows_for = [&](int st) __attribute__((always_inline)) {
    if constexpr (KV) stage_rows<D, W>(rows, st * kSI, ncols, row_of);
  };
  auto stage_dma_for = [&](int st, char *kd, char *ad, float *sd) __attribute__((always_inline)) {
    if constexpr (KV) stage_dma<D, true, KV, W>(rows, BK, ws.baug, ws.bs, kd, ad, sd, bank_row0, g.Mcap);
    else stage_dma_seq<D, true, W>(soff, c0 + st * kSI, BK.k, ws.baug, ws.bs, kd, ad, sd, bank_row0, g.Mcap);
  };
  // stage t in buffers (t % 3); rows of stage t + 2 loaded one step ahead
  auto step = [&](int t, const char *kb, const char *ab, const float *sb, char *kn, char *an, float *sn)
      __attribute__((always_inline)) {
    if (t + 1 < ns) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kOps));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
    stage_barrier();
    if (t + 2 < ns) {
      stage_dma_for(t + 2, kn, an, sn);
      if (t + 3 < ns) stage_rows_for(t + 3);
    }
    f32x16 u0, u1;
    stage_u<D, 0>(kb, ab, rf, u0, u1);
    const int nv0 = ncols - t * kSI;
    uint32_t sa;
    if (nv0 >= kSI) {
      epi(Full{}, u0, sb, kCT, sa);
      A64 += sa;
      epi(Full{}, u1, sb + kCT, kCT, sa);
      A64 += sa;
    } else {
      epi(Part{}, u0, sb, nv0, sa);
      A64 += sa;
      if (nv0 > kCT) {
        epi(Part{}, u1, sb + kCT, nv0 - kCT, sa);
        A64 += sa;
      }
    }
  };
  stage_rows_for(0);
  stage_dma_for(0, k0, a0, s0);
  if (ns > 1) {
    stage_rows_for(1);
    stage_dma_for(1, k1, a1, s1);
    if (ns > 2) stage_rows_for(2);
  }
  if constexpr (D <= 128) {
    // Tile-granular software pipeline (see tile_interleave).  Iteration t: tile 1
    // of stage t with the epilogue of tile 0 (the score scales of both tiles
    // read from stage t's buffer meanwhile); the wait for stage t + 1 and the
    // barrier; stage t + 3 issued into stage t's buffers; tile 0 of stage t + 1
    // with the epilogue of tile 1.
    int aoff[TileCfg<D>::kSteps];
    frag_offsets<D>(aoff);
    auto load_bs = [&](const float *tb, float (&bsv)[16]) __attribute__((always_inline)) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const float4 v = *reinterpret_cast<const float4 *>(&tb[8 * gq + 4 * h]);
        bsv[4 * gq + 0] = v.x;
        bsv[4 * gq + 1] = v.y;
        bsv[4 * gq + 2] = v.z;
        bsv[4 * gq + 3] = v.w;
      }
    };
    auto epi_full = [&](const f32x16 &u, const float (&bsv)[16]) __attribute__((always_inline)) -> uint32_t {
      uint32_t sa = 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float tt = FOLD ? u[i] : 1.0f + u[i];
        float tp = tt;
        if constexpr (P >= 2) tp = tt * tt;
        if constexpr (P == 4) tp = tp * tp;
        const float w = clamp_weight(rcp_rn(tp));
        sa += __float_as_uint(__builtin_fmaf(w, bsv[i], 8388608.0f));
      }
      return sa - 16u * kMagic;
    };
    f32x16 u;
    auto pstep = [&](int t, const char *kc, const char *ac, const float *sc, const char *kn, const char *an, char *kd,
                     char *ad, float *sd) __attribute__((always_inline)) {
      float b0[16], b1[16];
      load_bs(sc, b0);
      load_bs(sc + kCT, b1);
      f32x16 xx = tile_mfma<D>(kc, ac, 1, rf, aoff);
      uint32_t sa = epi_full(u, b0);
      tile_interleave<D, 11>();  // the 8 score-scale reads lead
      asm volatile("" : "+v"(sa));  // the epilogue of tile 0 stays beside the MFMAs of tile 1
      u = xx;
      if (t + 2 < ns) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kOps));
      else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      stage_barrier();
      if (t + 3 < ns) {
        stage_dma_for(t + 3, kd, ad, sd);
        if (t + 4 < ns) stage_rows_for(t + 4);
      }
      xx = tile_mfma<D>(kn, an, 0, rf, aoff);
      sa += epi_full(u, b1);
      tile_interleave<D>();
      u = xx;
      A64 += sa;
    };
    if (ns > 0) {
      if (ns > 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kOps));
      else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      stage_barrier();
      if (ns > 2) {
        stage_dma_for(2, k2, a2, s2);
        if (ns > 3) stage_rows_for(3);
      }
      u = tile_mfma<D>(k0, a0, 0, rf, aoff);
    }
    for (int t = 0; t + 1 < ns; t += 3) {
      pstep(t, k0, a0, s0, k1, a1, k0, a0, s0);
      if (t + 2 < ns) pstep(t + 1, k1, a1, s1, k2, a2, k1, a1, s1);
      if (t + 3 < ns) pstep(t + 2, k2, a2, s2, k0, a0, k2, a2, s2);
    }
    if (ns > 0) {  // the last stage (possibly partial): u holds its tile 0
      const int t = ns - 1;
      const int nv0 = ncols - t * kSI;
      // one call per buffer: the LDS arrays stay compile-time known
      auto last = [&](const char *kb, const char *ab, const float *sb) __attribute__((always_inline)) {
        uint32_t sa;
        epi(Part{}, u, sb, nv0, sa);
        A64 += sa;
        if (nv0 > kCT) {
          const f32x16 xx = tile_mfma<D>(kb, ab, 1, rf, aoff);
          epi(Part{}, xx, sb + kCT, nv0 - kCT, sa);
          A64 += sa;
        }
      };
      if (t % 3 == 0) last(k0, a0, s0);
      else if (t % 3 == 1) last(k1, a1, s1);
      else last(k2, a2, s2);
    }
  } else {
  for (int t = 0; t < ns; t += 3) {
    step(t, k0, a0, s0, k2, a2, s2);
    if (t + 1 < ns) step(t + 1, k1, a1, s1, k0, a0, s0);
    if (t + 2 < ns) step(t + 2, k2, a2, s2, k1, a1, s1);
  }
  }
  const uint64_t At = A64 + __shfl_xor(A64, 32, 64);
  if (!rv || h != 0) return;
  const size_t o = (size_t)b * g.N + x;
  atomicAdd(reinterpret_cast<unsigned long long *>(&ws.acol[o]), (unsigned long long)At);
}

// ---------------------------------------------------------------------------
// Row sums.  MODE selects rows, columns and where the sum goes.
// ---------------------------------------------------------------------------
enum RowSumMode { RS_CHUNK = 0, RS_FIXUP = 1, RS_SURV_EV = 2, RS_ADM_BASE = 3, RS_ADM_MUT = 4, RS_DENSITY = 5 };

constexpr int kChunksPerSplit = 1024 / kCkStride;   // RS_CHUNK: 1024 ordered candidates per workgroup
// Ordered candidates in the first part of the crossing search (whole chunks).
constexpr int kCrossFirst = 256;
static_assert(kCrossFirst % kCkStride == 0, "the first part ends on a chunk boundary");

// The three LDS stages of a Gram workgroup (separate arrays: with the stage
// known at compile time, reads of one stage never wait for loads into another).
template <int D>
struct StageBufs {
  char *k0, *k1, *k2, *a0, *a1, *a2;
  uint32_t *cb;  // [3][kSI] column sums of the stages (admitted x admitted only), or null
};

// DPP move (the partner lane's value) with a compile-time control.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
// Transposing reduction over the 16 lanes of a DPP row: the lane holds eight
// values a[i] (the first butterfly level already applied), returns the row
// sum for value index lane % 16.  Each level keeps the half of the values
// selected by one lane bit and adds the partner's copy of it: half-row mirror
// (bit 2), quad permutations (bits 1, 0).
__device__ __forceinline__ uint32_t row_transpose_tail(const uint32_t (&a)[8], int l) {
  uint32_t c[4], d[2];
  const bool b2 = (l >> 2) & 1, b1 = (l >> 1) & 1, b0 = l & 1;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t keep = b2 ? a[i + 4] : a[i], send = b2 ? a[i] : a[i + 4];
    c[i] = keep + dpp_mov<0x141>(send);  // row_half_mirror: lane 7 - x within 8 (bit 2 flipped)
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t keep = b1 ? c[i + 2] : c[i], send = b1 ? c[i] : c[i + 2];
    d[i] = keep + dpp_mov<0x4E>(send);  // quad_perm [2,3,0,1]: lane x ^ 2
  }
  const uint32_t keep = b0 ? d[1] : d[0], send = b0 ? d[0] : d[1];
  return keep + dpp_mov<0xB1>(send);  // quad_perm [1,0,3,2]: lane x ^ 1
}

// Body of one row-sum workgroup (bx, by, bz) = (row block, column split, bank).
template <int D, int P, int MODE, bool FOLD, bool KV>
__device__ __forceinline__ void rowsum_body(const dkv_bank &bank, const void *seg_k, const void *seg_v, const Geom &g,
                                            const Prm &p, const Workspace &ws, int64_t *out, int bx, int by, int bz,
                                            const StageBufs<D> &sb, int cfirst = 0, int clim = 1 << 30) {
  constexpr int W = gram_waves<D>();
  constexpr int kRowsPerWG = 32 * W;
  const int b = bz;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  const int m = ws.m[b];
  // descriptors: candidates, bank states, ordered candidates (stored concatenated)
  const Desc SK{static_cast<const uint16_t *>(seg_k), static_cast<const uint16_t *>(seg_v)};
  const Desc BK{static_cast<const uint16_t *>(bank.k), static_cast<const uint16_t *>(bank.v)};
  const Desc OK{ws.sk, nullptr};
  constexpr bool kNeedEv = MODE == RS_SURV_EV || MODE == RS_ADM_BASE || MODE == RS_ADM_MUT;
  const int n_ev = kNeedEv ? ws.n_ev[b] : 0;
  const int rs = (MODE == RS_FIXUP || kNeedEv) ? ws.r_star[b / g.gs] : 0;
  const int n_surv = m - n_ev;
  // rows
  int nrows;
  if constexpr (MODE == RS_CHUNK || MODE == RS_FIXUP || MODE == RS_DENSITY) nrows = m;
  else if constexpr (MODE == RS_SURV_EV) nrows = n_surv;
  else nrows = rs;
  if ((int)bx * kRowsPerWG >= nrows) return;
  // columns of this workgroup: [c0, c1) of the mode's column list
  int c0 = 0, c1 = 0;
  if constexpr (MODE == RS_CHUNK) {  // prefixes [cfirst, clim) of the order, 1,024 per split
    const int R = ws.R[b];
    c0 = cfirst + by * kChunksPerSplit * kCkStride;
    c1 = min(min(R, clim), c0 + kChunksPerSplit * kCkStride);
  } else if constexpr (MODE == RS_FIXUP) {
    c0 = (rs / kCkStride) * kCkStride;
    c1 = rs;
  } else {
    int total;
    if constexpr (MODE == RS_SURV_EV) total = n_ev;
    else if constexpr (MODE == RS_ADM_BASE) total = n_surv;
    else if constexpr (MODE == RS_ADM_MUT) total = rs;
    else total = m;
    // admitted x admitted: half splits, since a row block only takes the
    // columns from its own block on (finer work items balance the triangle)
    constexpr int kSplit = MODE == RS_ADM_MUT ? kColsPerSplit / 2 : kColsPerSplit;
    c0 = by * kSplit;
    c1 = min(total, c0 + kSplit);
  }
  // admitted x admitted is symmetric (W_xy = W_yx exactly, keys on the grid):
  // a workgroup takes the column stages from its own row block on; the diagonal
  // block gives row sums, every stage above it row and column sums
  constexpr bool kSym = MODE == RS_ADM_MUT;
  if constexpr (kSym) c0 = max(c0, (int)bx * kRowsPerWG);
  if (MODE != RS_FIXUP && c0 >= c1) return;  // the fix-up always writes rho~, even for r* % 256 == 0
  const int v = bx * kRowsPerWG + wave * 32 + n;
  const bool rv = v < nrows;
  // fix-up: rho~ = rho + the whole chunks before r* + (below) the partial chunk
  auto fixup_finish = [&](uint64_t tot) __attribute__((always_inline)) {
    // the two half-waves sum alternate 4-chunk groups
    const int full = rs / kCkStride;
    if (rv) {
      const uint4 *ckr = reinterpret_cast<const uint4 *>(ws.ck + (rb + v) * ws.nck);
      for (int c4 = h; 4 * c4 < full; c4 += 2) {
        const uint4 q = ckr[c4];
        const int c = 4 * c4;
        tot += (uint64_t)q.x + (c + 1 < full ? (uint64_t)q.y : 0) + (c + 2 < full ? (uint64_t)q.z : 0) +
               (c + 3 < full ? (uint64_t)q.w : 0);
      }
    }
    tot += __shfl_xor(tot, 32, 64);
    if (!rv || h != 0) return;
    const size_t row = rb + v;
    const int64_t rt = bank.rho[row] + (int64_t)tot;
    ws.rho_t[row] = rt;
    if (out) out[row] = rt;
  };
  if constexpr (MODE == RS_FIXUP) {
    // r* on a chunk boundary (uniform over the workgroup): no Gram, whole chunks only
    if (c0 >= c1) {
      fixup_finish(0);
      return;
    }
  }
  // row item
  Desc rsrc = BK;
  int64_t rrow = (int64_t)rb;
  float rnorm = 0.0f;
  size_t out_idx = 0;
  if (rv) {
    if constexpr (MODE == RS_CHUNK || MODE == RS_FIXUP || MODE == RS_DENSITY) {
      rrow = (int64_t)(rb + v);
      rnorm = bank.knorm[rb + v];
      out_idx = rb + v;
    } else if constexpr (MODE == RS_SURV_EV) {
      const int s = ws.surv_list[rb + v];
      rrow = (int64_t)(rb + s);
      rnorm = bank.knorm[rb + s];
      out_idx = rb + s;
    } else {
      const int x = ws.adm_list[nb + v];
      rsrc = SK;
      rrow = (int64_t)(nb + x);
      rnorm = ws.cnorm[nb + x];
      out_idx = nb + v;
    }
  }
  RowFrag<D> rf;
  load_row_frag<D, FOLD, KV>(rf, rsrc, rrow, rnorm, rv, -2.0f * p.inv_sigma2, p.inv_sigma2);
  // column items (absolute index j in the mode's list)
  auto row_of = [&](int j) -> int64_t {
    if constexpr (MODE == RS_CHUNK || MODE == RS_FIXUP) return (int64_t)(nb + j);
    else if constexpr (MODE == RS_SURV_EV) return (int64_t)(rb + ws.ev_list[rb + j]);
    else if constexpr (MODE == RS_ADM_BASE) return (int64_t)(rb + ws.surv_list[rb + j]);
    else if constexpr (MODE == RS_ADM_MUT) return (int64_t)(nb + ws.adm_list[nb + j]);
    else return (int64_t)(rb + j);
  };
  const Desc colbase = (MODE == RS_CHUNK || MODE == RS_FIXUP) ? OK : (MODE == RS_ADM_MUT ? SK : BK);
  // the ordered candidates are stored as whole descriptors; the others are split for [K; V]
  constexpr bool kColSplit = KV && !(MODE == RS_CHUNK || MODE == RS_FIXUP);
  const uint4 *colaug = (MODE == RS_CHUNK || MODE == RS_FIXUP) ? ws.saug : (MODE == RS_ADM_MUT ? ws.caug : ws.baug);
  // the column rows lie in bank b's candidates or in its slots
  constexpr bool kColCand = MODE == RS_CHUNK || MODE == RS_FIXUP || MODE == RS_ADM_MUT;
  const int64_t col_row0 = kColCand ? (int64_t)nb : (int64_t)rb;
  const int col_nrows = kColCand ? g.N : g.Mcap;  // rows of that region
  constexpr bool kDiag = (MODE == RS_ADM_MUT || MODE == RS_DENSITY);
  // fragment reads kept ahead of the MFMAs where the registers allow it
  constexpr int kStageAhead = (D <= 128 && (MODE == RS_CHUNK || MODE == RS_FIXUP || MODE == RS_DENSITY)) ? 4 : 0;
  // the prefix-chunk Gram runs software-pipelined (below)
  constexpr bool kPipe = MODE == RS_CHUNK && D <= 128;
  uint64_t S64 = 0;
  uint32_t chunk_sum = 0;
  const int ncols = c1 - c0;
  const int ns = (ncols + kSI - 1) / kSI;
  auto row_of_rel = [&](int j) -> int64_t { return row_of(c0 + j); };
  const int wg_row0 = bx * kRowsPerWG;
  // sum of the lane's 16 weights of one 32-column tile starting at list index j0
  auto tile_sum = [&](const f32x16 &u, int j0, int nvalid) __attribute__((always_inline)) -> uint32_t {
    const bool diag_tile = kDiag && (j0 < wg_row0 + kRowsPerWG) && (j0 + kCT > wg_row0);
    if (nvalid >= kCT && !diag_tile) return lane_wsum<P, false, FOLD>(u, kCT, h);
    uint32_t sm = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int mm = col_of_reg(q, h);
      uint32_t raw = weight_raw<P, FOLD>(u[q], 8388608.0f);
      bool ok = mm < nvalid;
      if (kDiag) ok = ok && (j0 + mm != v);
      sm += ok ? raw : kMagic;
    }
    return sm - 16u * kMagic;
  };
  // column sums of one 32-column tile above the diagonal block: every lane's 16
  // weights (masked rows and columns as zero), the row partials by DPP
  // butterfly, and one LDS add per lane (the two rows of each half-wave add
  // partials of the same 16 columns); returns the lane's row sum
  const bool rows_full = wg_row0 + kRowsPerWG <= nrows;
  auto sym_tile = [&](const f32x16 &u, int nvalid, uint32_t *cb, int off) __attribute__((always_inline)) -> uint32_t {
    const bool full = nvalid >= kCT && rows_full;
    const bool b3 = (l >> 3) & 1;
    uint32_t a[8], rsum = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      // values i and i + 8, then the first butterfly level (row mirror: lane
      // 15 - x, bit 3 flipped)
      uint32_t r0 = weight_raw<P, FOLD>(u[i], 8388608.0f), r1 = weight_raw<P, FOLD>(u[i + 8], 8388608.0f);
      if (!full) {
        r0 = (rv && col_of_reg(i, h) < nvalid) ? r0 : kMagic;
        r1 = (rv && col_of_reg(i + 8, h) < nvalid) ? r1 : kMagic;
      }
      rsum += r0 + r1;
      const uint32_t keep = b3 ? r1 : r0, send = b3 ? r0 : r1;
      a[i] = keep + dpp_mov<0x140>(send);
    }
    const uint32_t csum = row_transpose_tail(a, l) - 16u * kMagic;
    atomicAdd(&cb[off + col_of_reg(l & 15, h)], csum);
    return rsum - 16u * kMagic;
  };
  // column sums of stage t (whose adds finished before the barrier just passed)
  // to the global sums; the buffer is cleared for stage t + 3
  auto flush_cols = [&](int t) __attribute__((always_inline)) {
    const int j0 = c0 + t * kSI;
    if (j0 < wg_row0 + kRowsPerWG || l >= kSI / W) return;
    uint32_t *cb = sb.cb + (t % 3) * kSI;
    const int idx = wave * (kSI / W) + l;
    const uint32_t val = cb[idx];
    cb[idx] = 0;
    if (j0 + idx < c1 && val != 0)
      atomicAdd(reinterpret_cast<unsigned long long *>(&ws.mut_adm[nb + j0 + idx]), (unsigned long long)val);
  };
  constexpr int kOps = stage_ops<D, false, W>();
  // Stage t in buffers t % 3.  The global rows of stage t + 2 were fetched one
  // step earlier (list lookups for the maintenance stages), so issuing its
  // loads never waits for the loads still in flight.
  // Two row sets used alternately (the loop is unrolled 6 = lcm(3, 2) times),
  // so that no register copy waits for a lookup still in flight.
  StageRows<D, W> rowsA, rowsB;
  using Rows = StageRows<D, W>;
  // stage s covers list entries c0 + s kSI ..; where those are consecutive rows
  // of one region (ordered candidates, bank slots in order) and whole-row
  // descriptors, the loads take the per-lane offsets of consecutive rows and no
  // row list is built
  constexpr bool kSeqRows = !kColSplit && (MODE == RS_CHUNK || MODE == RS_FIXUP || MODE == RS_DENSITY);
  [[maybe_unused]] const StageOff<D, W> soff = stage_offsets<D, W>();
  auto stage_rows_for = [&](Rows &r, int st) __attribute__((always_inline)) {
    if constexpr (!kSeqRows) stage_rows<D, W>(r, st * kSI, ncols, row_of_rel);
  };
  auto stage_dma_for = [&](const Rows &r, int st, char *kd, char *ad) __attribute__((always_inline)) {
    if constexpr (kSeqRows)
      stage_dma_seq<D, false, W>(soff, c0 + st * kSI, colbase.k, colaug, nullptr, kd, ad, nullptr, col_row0, col_nrows);
    else stage_dma<D, false, kColSplit, W>(r, colbase, colaug, nullptr, kd, ad, nullptr, col_row0, col_nrows);
  };
  auto step = [&](int t, const char *kb, const char *ab, char *kn, char *an, Rows &use, Rows &fill)
      __attribute__((always_inline)) {
    if (t + 1 < ns) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kOps));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
    stage_barrier();
    if (t + 2 < ns) {
      if (t + 3 < ns) stage_rows_for(fill, t + 3);
      stage_dma_for(use, t + 2, kn, an);
    }
    if constexpr (kSym) {
      if (t > 0) flush_cols(t - 1);
    }
    f32x16 u0, u1;
    stage_u<D, kStageAhead>(kb, ab, rf, u0, u1);
    const int nv0 = ncols - t * kSI;
    const int j0 = c0 + t * kSI;
    uint32_t s2;
    if (kSym && j0 >= wg_row0 + kRowsPerWG) {
      uint32_t *cb = sb.cb + (t % 3) * kSI;
      s2 = sym_tile(u0, nv0, cb, 0);
      if (nv0 > kCT) s2 += sym_tile(u1, nv0 - kCT, cb, kCT);
    } else {
      s2 = tile_sum(u0, j0, nv0);
      if (nv0 > kCT) s2 += tile_sum(u1, j0 + kCT, nv0 - kCT);
    }
    if constexpr (MODE == RS_CHUNK) {
      chunk_sum += s2;
      const bool chunk_end = ((t + 1) % (kCkStride / kSI)) == 0 || t + 1 == ns;
      if (chunk_end) {
        const uint32_t tot = chunk_sum + __shfl_xor(chunk_sum, 32, 64);
        if (rv && h == 0) ws.ck[(rb + v) * ws.nck + (j0 / kCkStride)] = tot;
        chunk_sum = 0;
      }
    } else {
      S64 += s2;
    }
  };
  if constexpr (kSym) {
    // cleared before the first stage barrier
    for (int i = threadIdx.x; i < 3 * kSI; i += 64 * W) sb.cb[i] = 0;
  }
  if (ns > 0) {
    stage_rows_for(rowsA, 0);
    stage_dma_for(rowsA, 0, sb.k0, sb.a0);
    if (ns > 1) {
      stage_rows_for(rowsB, 1);
      stage_dma_for(rowsB, 1, sb.k1, sb.a1);
      if (ns > 2) stage_rows_for(rowsA, 2);
    }
  }
  if constexpr (kPipe) {
    // Software pipeline of the prefix-chunk Gram at the granularity of one
    // 32-column tile: the MFMAs of the next tile run interleaved with the
    // epilogue of the current one, so that one wave keeps the matrix cores and
    // the VALU busy at the same time.  Stage s (tiles 2 s, 2 s + 1) uses
    // buffers s % 3 and rows (s even ? rowsA : rowsB).  Iteration t: tile 1
    // of stage t with the epilogue of tile 0; then the wait for stage t + 1,
    // the barrier (every wave is done with the buffers of stage t), stage t + 3
    // issued into them, and tile 0 of stage t + 1 with the epilogue of tile 1.
    static_assert(kCkStride == kSI, "one prefix chunk per stage");
    int aoff[TileCfg<D>::kSteps];
    frag_offsets<D>(aoff);
    auto tile_mfma_ = [&](const char *kb, const char *ab, int half) __attribute__((always_inline)) -> f32x16 {
      return tile_mfma<D>(kb, ab, half, rf, aoff);
    };
    auto store_chunk = [&](int t, uint32_t s2) __attribute__((always_inline)) {
      const uint32_t tot = s2 + __shfl_xor(s2, 32, 64);
      if (rv && h == 0) ws.ck[(rb + v) * ws.nck + ((c0 + t * kSI) / kCkStride)] = tot;
    };
    f32x16 u;
    // iteration t for a full stage t that is not the last
    auto pstep = [&](int t, const char *kc, const char *ac, const char *kn, const char *an, char *kd, char *ad,
                     Rows &use, Rows &fill) __attribute__((always_inline)) {
      f32x16 x = tile_mfma_(kc, ac, 1);
      uint32_t s2 = lane_wsum<P, false, FOLD>(u, kCT, h);
      tile_interleave<D>();
      asm volatile("" : "+v"(s2));  // the epilogue of tile 0 stays beside the MFMAs of tile 1
      u = x;
      if (t + 2 < ns) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kOps));
      else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      stage_barrier();
      if (t + 3 < ns) {
        if (t + 4 < ns) stage_rows_for(fill, t + 4);
        stage_dma_for(use, t + 3, kd, ad);
      }
      x = tile_mfma_(kn, an, 0);
      s2 += lane_wsum<P, false, FOLD>(u, kCT, h);
      tile_interleave<D>();
      u = x;
      store_chunk(t, s2);
    };
    if (ns > 0) {
      if (ns > 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kOps));
      else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      stage_barrier();
      if (ns > 2) {
        if (ns > 3) stage_rows_for(rowsB, 3);
        stage_dma_for(rowsA, 2, sb.k2, sb.a2);
      }
      u = tile_mfma_(sb.k0, sb.a0, 0);
    }
    // iteration t: stage t in buffers t % 3, stage t + 1 in (t + 1) % 3, stage t + 3
    // issued into t % 3 with rows (t odd ? rowsA : rowsB), rows of t + 4 fetched
    for (int t = 0; t + 1 < ns; t += 6) {
      pstep(t, sb.k0, sb.a0, sb.k1, sb.a1, sb.k0, sb.a0, rowsB, rowsA);
      if (t + 2 < ns) pstep(t + 1, sb.k1, sb.a1, sb.k2, sb.a2, sb.k1, sb.a1, rowsA, rowsB);
      if (t + 3 < ns) pstep(t + 2, sb.k2, sb.a2, sb.k0, sb.a0, sb.k2, sb.a2, rowsB, rowsA);
      if (t + 4 < ns) pstep(t + 3, sb.k0, sb.a0, sb.k1, sb.a1, sb.k0, sb.a0, rowsA, rowsB);
      if (t + 5 < ns) pstep(t + 4, sb.k1, sb.a1, sb.k2, sb.a2, sb.k1, sb.a1, rowsB, rowsA);
      if (t + 6 < ns) pstep(t + 5, sb.k2, sb.a2, sb.k0, sb.a0, sb.k2, sb.a2, rowsA, rowsB);
    }
    // the last stage (possibly partial); u holds its tile 0
    if (ns > 0) {
      const int t = ns - 1;
      const int nv0 = ncols - t * kSI;
      const int j0 = c0 + t * kSI;
      uint32_t s2 = tile_sum(u, j0, nv0);
      if (nv0 > kCT) {
        // one call per buffer: the LDS arrays stay compile-time known (no generic pointers)
        f32x16 x;
        if (t % 3 == 0) x = tile_mfma_(sb.k0, sb.a0, 1);
        else if (t % 3 == 1) x = tile_mfma_(sb.k1, sb.a1, 1);
        else x = tile_mfma_(sb.k2, sb.a2, 1);
        s2 += tile_sum(x, j0 + kCT, nv0 - kCT);
      }
      store_chunk(t, s2);
    }
    return;
  }
  // step t issues stage t + 2 with the rows fetched at step t - 1 and fetches
  // those of stage t + 3: stage t + 2 uses rowsA when t is even
  for (int t = 0; t < ns; t += 6) {
    step(t, sb.k0, sb.a0, sb.k2, sb.a2, rowsA, rowsB);
    if (t + 1 < ns) step(t + 1, sb.k1, sb.a1, sb.k0, sb.a0, rowsB, rowsA);
    if (t + 2 < ns) step(t + 2, sb.k2, sb.a2, sb.k1, sb.a1, rowsA, rowsB);
    if (t + 3 < ns) step(t + 3, sb.k0, sb.a0, sb.k2, sb.a2, rowsB, rowsA);
    if (t + 4 < ns) step(t + 4, sb.k1, sb.a1, sb.k0, sb.a0, rowsA, rowsB);
    if (t + 5 < ns) step(t + 5, sb.k2, sb.a2, sb.k1, sb.a1, rowsB, rowsA);
  }
  if constexpr (kSym) {
    if (ns > 0) {
      __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      stage_barrier();
      flush_cols(ns - 1);
    }
  }
  if constexpr (MODE == RS_CHUNK) return;
  if constexpr (MODE == RS_FIXUP) {
    fixup_finish(S64);
    return;
  }
  uint64_t tot = S64;
  tot += __shfl_xor(tot, 32, 64);
  if (!rv || h != 0) return;
  {
    int64_t *dst = (MODE == RS_SURV_EV || MODE == RS_DENSITY) ? ws.sub : (MODE == RS_ADM_BASE ? ws.sub_adm : ws.mut_adm);
    atomicAdd(reinterpret_cast<unsigned long long *>(&dst[out_idx]), (unsigned long long)tot);
  }
}

template <int D, int P, int MODE, bool FOLD, bool KV>
__global__ __launch_bounds__(64 * gram_waves<D>(), gram_waves<D>() == 4 ? 3 : 2) void k_rowsum_mfma(
    dkv_bank bank, const void *seg_k, const void *seg_v, Geom g, Prm p, Workspace ws, int64_t *out) {
  constexpr int KB = SCfg<D>::KEYB, AB = SCfg<D>::AUGB;
  __shared__ __attribute__((aligned(1024))) char k0[KB], k1[KB], k2[KB];
  __shared__ __attribute__((aligned(16))) char a0[AB], a1[AB], a2[AB];
  const StageBufs<D> sb{k0, k1, k2, a0, a1, a2, nullptr};
  rowsum_body<D, P, MODE, FOLD, KV>(bank, seg_k, seg_v, g, p, ws, out, blockIdx.x, blockIdx.y, blockIdx.z, sb);
}

// Maintenance work items (Supp. C): per bank, the (row block, column split)
// pairs of its three Grams that hold pairs: survivors x evicted (row blocks of
// the survivors x splits of the evicted), admitted x survivors, and admitted x
// admitted (half splits).  A bank that admits nothing and releases nothing
// has none.
struct MaintItems {
  int rows_s, rows_a, n_se, n_ab, n_am;
};
// rpw: rows per workgroup of the maintenance Grams
__device__ __forceinline__ MaintItems maint_items(const Geom &g, const Workspace &ws, int b, int rpw) {
  const int ne = ws.n_ev[b], rs = ws.r_star[b / g.gs], ns = ws.m[b] - ne;
  MaintItems it;
  it.rows_s = (ns + rpw - 1) / rpw;
  it.rows_a = (rs + rpw - 1) / rpw;
  it.n_se = it.rows_s * ((ne + kColsPerSplit - 1) / kColsPerSplit);
  it.n_ab = it.rows_a * ((ns + kColsPerSplit - 1) / kColsPerSplit);
  it.n_am = it.rows_a * ((rs + kColsPerSplit / 2 - 1) / (kColsPerSplit / 2));
  return it;
}

// Exclusive prefix of the banks' work item counts (one workgroup).
constexpr int kPlanThreads = 1024;
constexpr unsigned kMaintWgs = 4096;  // maintenance workgroups (3 per CU on 256 CUs, over 5 rounds)
__global__ __launch_bounds__(kPlanThreads) void k_maint_plan(Geom g, Workspace ws, int rpw) {
  __shared__ int32_t part[kPlanThreads];
  int carry = 0;
  for (int b0 = 0; b0 < g.B; b0 += kPlanThreads) {
    const int b = b0 + (int)threadIdx.x;
    int cnt = 0;
    if (b < g.B) {
      const MaintItems it = maint_items(g, ws, b, rpw);
      cnt = it.n_se + it.n_ab + it.n_am;
    }
    part[threadIdx.x] = cnt;
    __syncthreads();
    for (int o = 1; o < kPlanThreads; o <<= 1) {  // inclusive scan
      const int y = threadIdx.x >= (unsigned)o ? part[threadIdx.x - o] : 0;
      __syncthreads();
      part[threadIdx.x] += y;
      __syncthreads();
    }
    if (b < g.B) ws.maint_off[b] = carry + part[threadIdx.x] - cnt;
    carry += part[kPlanThreads - 1];
    __syncthreads();
  }
  if (threadIdx.x == 0) ws.maint_off[g.B] = carry;
}

// The maintenance Grams of every bank over the planned work items: workgroup
// k takes the items [k per, (k + 1) per) in bank order, per = total / grid
// rounded up, so a frozen block (no item) costs one read per workgroup.
template <int D, int P, bool FOLD, bool KV>
__global__ __launch_bounds__(64 * gram_waves<D>(), gram_waves<D>() == 4 ? 3 : 2) void k_maint_mfma(
    dkv_bank bank, const void *seg_k, const void *seg_v, Geom g, Prm p, Workspace ws) {
  constexpr int kRpw = 32 * gram_waves<D>();
  constexpr int KB = SCfg<D>::KEYB, AB = SCfg<D>::AUGB;
  __shared__ __attribute__((aligned(1024))) char k0[KB], k1[KB], k2[KB];
  __shared__ __attribute__((aligned(16))) char a0[AB], a1[AB], a2[AB];
  __shared__ __attribute__((aligned(16))) uint32_t cb[3 * kSI];
  const StageBufs<D> sb{k0, k1, k2, a0, a1, a2, cb};
  const int total = ws.maint_off[g.B];
  const int per = (total + (int)gridDim.x - 1) / (int)gridDim.x;
  const int w0 = (int)blockIdx.x * per, w1 = min(total, w0 + per);
  if (w0 >= w1) return;
  // bank of item w0: the last bank whose first item is <= w0 (banks without
  // items share the offset of the next bank)
  int lo = 0, hi = g.B;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (ws.maint_off[mid] <= w0) lo = mid;
    else hi = mid;
  }
  int b = lo, i = w0 - ws.maint_off[b];
  MaintItems it = maint_items(g, ws, b, kRpw);
  for (int w = w0; w < w1; ++w, ++i) {
    while (i >= it.n_se + it.n_ab + it.n_am && b + 1 < g.B) {  // next bank with items
      i -= it.n_se + it.n_ab + it.n_am;
      it = maint_items(g, ws, ++b, kRpw);
    }
    __syncthreads();  // the previous item's LDS stages are done with
    if (i < it.n_se) {
      rowsum_body<D, P, RS_SURV_EV, FOLD, KV>(bank, seg_k, seg_v, g, p, ws, nullptr, i % it.rows_s, i / it.rows_s, b,
                                          sb);
    } else if (i < it.n_se + it.n_ab) {
      const int j = i - it.n_se;
      rowsum_body<D, P, RS_ADM_BASE, FOLD, KV>(bank, seg_k, seg_v, g, p, ws, nullptr, j % it.rows_a, j / it.rows_a, b,
                                           sb);
    } else {
      const int j = i - it.n_se - it.n_ab;
      rowsum_body<D, P, RS_ADM_MUT, FOLD, KV>(bank, seg_k, seg_v, g, p, ws, nullptr, j % it.rows_a, j / it.rows_a, b,
                                          sb);
    }
  }
}

// ---------------------------------------------------------------------------
// First violating prefix length of every bank state (Eqs. 8-9).
//
// Chunk search: the state's group of 8 lanes holds its 64-candidate chunk
// sums, 16 per lane; a scan over the group gives every lane's prefix, and the
// lane whose 16 chunks contain the first prefix that lifts rho + P to tau b
// (2^k (rho + P) >= T b, integers) finds the chunk and how much of that
// chunk's weight is still needed.  Then the exact length inside the chunk,
// with the same binary32 weights.  States that never reach the bound within
// the tested prefixes get R + 1; states whose empty prefix already violates 0.
// ---------------------------------------------------------------------------
constexpr int kCrossLanes = 8;                      // lanes per state in the chunk search
constexpr int kCrossPerLane = 16;                   // chunk sums per lane
constexpr int kCrossStates = 64 / kCrossLanes;      // states per chunk-search pass of a wave

// v of the lane O below within a group of 8 lanes (a DPP row shift: the group
// lies in one row of 16 lanes), 0 for the group's first O lanes (q < O).  A DPP
// read from a lane that is switched off returns 0, so the shift runs with every
// lane on (the empty asm keeps it out of the branch of q >= O) and the select
// follows.
template <int O>
__device__ __forceinline__ uint64_t group_shr_u64(uint64_t v, int q) {
  static_assert(O >= 1 && O < kCrossLanes, "shift within a group");
  uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, 0x110 + O, 0xF, 0xF, true);
  uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), 0x110 + O, 0xF, 0xF, true);
  asm volatile("" : "+v"(lo), "+v"(hi));
  return q >= O ? ((uint64_t)hi << 32) | lo : 0ull;
}

struct CrossFind {
  bool pos;       // the bound lies above rho (else the empty prefix violates)
  bool hit;       // this lane's chunks hold the first prefix that reaches it
  int ch;         // that chunk (hit lane only)
  uint32_t need;  // the bound minus rho minus every chunk before it, in [1, 2^29] (hit lane only)
};

// Chunk search for one bank row by lane q of its group: the loads (issued
// together for several rows), then the search; nch chunks are tested.
struct CrossRow {
  int64_t base, rho;
  uint4 x[kCrossPerLane / 4];
};

__device__ __forceinline__ CrossRow cross_load(const dkv_bank &bank, const Workspace &ws, size_t row, int q, int nch) {
  CrossRow r;
  r.base = bank.base[row];
  r.rho = bank.rho[row];
  // 16-byte groups of the row (nck >= 4, a multiple of 4, at least nch); only
  // those that hold tested chunks are read (the rest may be stale), clamped
  const uint4 *ckr = reinterpret_cast<const uint4 *>(ws.ck + row * ws.nck);
  const int last = ws.nck / 4 - 1;
#pragma unroll
  for (int v4 = 0; v4 < kCrossPerLane / 4; ++v4) {
    const int grp = (kCrossPerLane * q) / 4 + v4;
    r.x[v4] = 4 * grp < nch ? ckr[min(grp, last)] : uint4{0u, 0u, 0u, 0u};
  }
  return r;
}

__device__ __forceinline__ CrossFind cross_find(const CrossRow &r, const Prm &p, int nch, int q) {
  static_assert((DKV_MAX_CANDIDATES + kCkStride - 1) / kCkStride <= kCrossLanes * kCrossPerLane,
                "every chunk sum of a state is held by its lane group");
  const int64_t lim = ((int64_t)p.tau_num * r.base + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
  const int64_t thr = lim - r.rho;
  uint32_t c[kCrossPerLane];
#pragma unroll
  for (int v4 = 0; v4 < kCrossPerLane / 4; ++v4) {
    const int c0 = kCrossPerLane * q + 4 * v4;
    c[4 * v4 + 0] = c0 + 0 < nch ? r.x[v4].x : 0u;
    c[4 * v4 + 1] = c0 + 1 < nch ? r.x[v4].y : 0u;
    c[4 * v4 + 2] = c0 + 2 < nch ? r.x[v4].z : 0u;
    c[4 * v4 + 3] = c0 + 3 < nch ? r.x[v4].w : 0u;
  }
  // a chunk sum is at most 64 x 2^23 = 2^29: seven of them fit 32 bits, eight may not
  uint32_t a7 = 0, b7 = 0;
#pragma unroll
  for (int t = 0; t < 7; ++t) {
    a7 += c[t];
    b7 += c[8 + t];
  }
  const uint64_t s8a = (uint64_t)a7 + c[7], tot = s8a + (uint64_t)b7 + c[15];
  // inclusive scan over the group (DPP row shifts: a group of 8 lies in one row of 16 lanes)
  uint64_t incl = tot;
  incl += group_shr_u64<1>(incl, q);
  incl += group_shr_u64<2>(incl, q);
  incl += group_shr_u64<4>(incl, q);
  // what this lane's chunks must still supply; the crossing lies in them iff it is in (0, tot]
  const int64_t need_l = thr - (int64_t)(incl - tot);
  CrossFind f;
  f.pos = thr > 0;
  f.hit = f.pos && need_l > 0 && need_l <= (int64_t)tot;
  // the half of the lane's chunks that holds it, and the rest in [1, 2^32] (32 bits after -1)
  const bool hi = need_l > (int64_t)s8a;
  const uint32_t nd1 = (uint32_t)((uint64_t)(hi ? need_l - (int64_t)s8a : need_l) - 1u);
  // chunks of that half before the crossing: those whose end prefix is still below the bound
  // (the half's full sum reaches it, so at most seven, whose prefixes fit 32 bits)
  uint32_t pr = 0, pre = 0;
  int cnt = 0;
#pragma unroll
  for (int t = 0; t < 7; ++t) {
    pr += hi ? c[8 + t] : c[t];
    if (pr <= nd1) {
      ++cnt;
      pre = pr;
    }
  }
  f.ch = kCrossPerLane * q + (hi ? 8 : 0) + cnt;
  f.need = nd1 - pre + 1u;
  return f;
}

// The whole crossing search over every tested prefix, for the groups that the
// first part leaves open (every group when first crossings are requested).
// A wave takes 32 states, a workgroup 128.
// The chunk search runs in four passes of eight states; each state's result then
// moves to lanes n and n + 32 (n = its index in the wave).  The exact walk: the
// workgroup's crossing chunks, in increasing order, each staged through LDS as a
// column stage of the Gram kernels (two buffers, alternating), and in every wave
// that has a state crossing there one 64 x 32 MFMA Gram with the Gram stages' own
// tiles: A = the chunk's ordered candidates (two tiles of 32) with their norm
// steps, B = the 32 states as row items, so lane (n, h) gets t of state n with
// candidates 8 k + 4 h + j (registers 4 k + j) of each tile, bit for bit the t
// that made the chunk sums; each lane keeps the Gram of its own chunk.  Then,
// once per lane, the weights summed in candidate order (the two halves exchange
// their 4-candidate group sums), and the crossing length is one plus the number
// of candidates whose inclusive prefix is still below the need.
constexpr int kCrossWaveStates = 32;

template <int D, int P, bool FOLD, bool KV>
__global__ __launch_bounds__(64 * kWaves, D <= 128 ? 3 : 2) void k_cross_mfma(dkv_bank bank, Geom g, Prm p, Workspace ws,
                                                                            int32_t *out_first) {
  static_assert(kCkStride == 64, "two 32-candidate tiles per chunk");
  constexpr int KSW = D / 16;
  const int b = blockIdx.y;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int grp = l / kCrossLanes, q = l % kCrossLanes, n32 = l & 31, hw = l >> 5;
  const int i0 = (blockIdx.x * kWaves + wave) * kCrossWaveStates;
  const int m = ws.m[b], R = ws.R[b];
  if (!ws.more[b / g.gs]) return;  // the first part decided this group
  if ((int)blockIdx.x * kWaves * kCrossWaveStates >= m) return;  // whole workgroup (the walk has barriers)
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  const int nch = (R + kCkStride - 1) / kCkStride;
  // per state of this lane's column: whether its bound lies above rho, whether
  // it crosses within the tested prefixes, the crossing chunk and the need
  int my_ch = 0;
  uint32_t my_need = 0;
  bool my_pos = false, my_walk = false;
  constexpr int kPasses = kCrossWaveStates / kCrossStates;
  CrossRow rows[kPasses];  // every pass's loads in flight together
#pragma unroll
  for (int ps = 0; ps < kPasses; ++ps)
    rows[ps] = cross_load(bank, ws, rb + min(i0 + kCrossStates * ps + grp, m - 1), q, nch);
#pragma unroll
  for (int ps = 0; ps < kPasses; ++ps) {
    const int s = kCrossStates * ps + grp;
    const bool valid = i0 + s < m;
    const CrossFind f = cross_find(rows[ps], p, nch, q);
    const unsigned long long pos = __ballot(valid && f.pos);
    const unsigned long long hits = __ballot(valid && f.hit);
    // group g8 of this pass -> lanes n32 = 8 ps + g8
    const int g8 = (n32 - kCrossStates * ps) & (kCrossStates - 1);
    const unsigned gbits = (unsigned)(hits >> (kCrossLanes * g8)) & 0xFFu;
    const int src = kCrossLanes * g8 + (gbits ? __ffs(gbits) - 1 : 0);
    const int ch = __shfl(f.ch, src, 64);
    const uint32_t nd = __shfl(f.need, src, 64);
    if ((n32 >> 3) == ps) {
      my_ch = ch;
      my_need = nd;
      my_pos = (pos >> (kCrossLanes * g8)) & 1ull;
      my_walk = gbits != 0;
    }
  }
  int first = my_pos ? R + 1 : 0;
  // the workgroup's crossing chunks (at most 128: four words)
  __shared__ uint32_t chunk_set[4];
  if (threadIdx.x < 4) chunk_set[threadIdx.x] = 0;
  __syncthreads();
  if (my_walk && hw == 0) atomicOr(&chunk_set[my_ch >> 5], 1u << (my_ch & 31));
  __syncthreads();
  uint32_t cs[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) cs[k] = __builtin_amdgcn_readfirstlane(chunk_set[k]);
  if (cs[0] | cs[1] | cs[2] | cs[3]) {  // uniform over the workgroup
    // B operand: this lane's state as the Gram stages hold a row item (keys
    // times -2 / sigma^2 and the norm step); read for the states that walk only
    // (the others' columns of the Gram are not used)
    const int64_t srow = (int64_t)(rb + min(i0 + n32, m - 1));
    RowFrag<D> rf;
    load_row_frag<D, FOLD, KV>(rf, Desc{static_cast<const uint16_t *>(bank.k), static_cast<const uint16_t *>(bank.v)},
                               srow, my_walk ? bank.knorm[srow] : 0.0f, my_walk, -2.0f * p.inv_sigma2, p.inv_sigma2);
    int aoff[TileCfg<D>::kSteps];
    frag_offsets<D>(aoff);
    // each crossing chunk's 64 ordered candidates go through a stage buffer
    // (two, alternating) exactly as in the chunk-sum Gram, so t and every
    // weight are those of the chunk sums bit for bit; each lane keeps the
    // Gram of its own chunk
    constexpr int KB = SCfg<D>::KEYB, AB = SCfg<D>::AUGB;
    __shared__ __attribute__((aligned(1024))) char kbuf[2][KB];
    __shared__ __attribute__((aligned(16))) char abuf[2][AB];
    const Desc OK{ws.sk, nullptr};
    const StageOff<D> soff = stage_offsets<D>();
    auto issue = [&](int c, int buf) __attribute__((always_inline)) {
      stage_dma_seq<D, false>(soff, c * kCkStride, OK.k, ws.saug, nullptr, kbuf[buf], abuf[buf], nullptr, (int64_t)nb,
                              g.N);
    };
    // the chunks in increasing order (uniform over the workgroup)
    auto pop_chunk = [&]() __attribute__((always_inline)) -> int {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (cs[k]) {
          const int c = 32 * k + __builtin_ctz(cs[k]);
          cs[k] &= cs[k] - 1;
          return c;
        }
      return -1;
    };
    f32x16 mine[2] = {};
    bool partial = false;
    int c = pop_chunk(), buf = 0;
    issue(c, 0);
    while (c >= 0) {
      __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      stage_barrier();  // every wave's loads of chunk c landed; every wave is done with the other buffer
      const int cn = pop_chunk();
      if (cn >= 0) issue(cn, buf ^ 1);
      partial = partial || (c + 1) * kCkStride > R;
      const bool keep = my_walk && my_ch == c;
      if (__ballot(keep)) {  // uniform over the wave
#pragma unroll
        for (int tl = 0; tl < 2; ++tl) {
          const f32x16 x = tile_mfma<D>(kbuf[buf], abuf[buf], tl, rf, aoff);
#pragma unroll
          for (int r = 0; r < 16; ++r) mine[tl][r] = keep ? x[r] : mine[tl][r];
        }
      }
      c = cn;
      buf ^= 1;
    }
    // weights in candidate order inside the lane (groups of four consecutive
    // candidates, k = 0..3 of each tile, the two halves alternating); candidates
    // past R weigh nothing (wave-uniform test: a chunk that ends past R)
    const int ch0 = my_ch * kCkStride;
    const int nvalid = min(kCkStride, R - ch0);
    uint32_t w[2][16], gs[2][4];
    auto weights = [&](auto mask_tag) __attribute__((always_inline)) {
      constexpr bool MASK = decltype(mask_tag)::value;
#pragma unroll
      for (int tl = 0; tl < 2; ++tl) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          gs[tl][k] = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            uint32_t W = weight_raw<P, FOLD>(mine[tl][4 * k + j], 8388608.0f) - kMagic;
            if constexpr (MASK) {
              asm volatile("" : "+v"(W));  // computed for every lane, then masked
              W = 32 * tl + 8 * k + 4 * hw + j < nvalid ? W : 0u;
            }
            w[tl][4 * k + j] = W;
            gs[tl][k] += W;
          }
        }
      }
    };
    if (!__ballot(my_walk)) goto done;  // uniform over the wave
    if (partial) weights(std::integral_constant<bool, true>{});
    else weights(std::integral_constant<bool, false>{});
    // inclusive prefixes in candidate order; the crossing length is one plus the
    // number still below the need.  Candidates past R add nothing, so their
    // prefix equals the last valid one's and they are counted only if that one
    // was (cnt then reaches nvalid either way).
    uint32_t run = 0, cnt = 0;
    const uint32_t nd1 = my_need - 1u;
#pragma unroll
    for (int tl = 0; tl < 2; ++tl) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t other = __shfl_xor(gs[tl][k], 32, 64);
        uint32_t pr = run + (hw ? other : 0u);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          pr += w[tl][4 * k + j];
          cnt += pr <= nd1 ? 1u : 0u;
        }
        run += gs[tl][k] + other;
      }
    }
    cnt += __shfl_xor(cnt, 32, 64);
    if (my_walk) first = (int)cnt < nvalid ? ch0 + (int)cnt + 1 : ch0 + nvalid;  // the latter unreachable
  }
done:
  const int i = i0 + n32;
  if (hw == 0 && i < m) {
    ws.first[rb + i] = first;
    if (out_first) out_first[rb + i] = first;
  }
}

// The first part of the crossing search in one pass: the prefix-chunk Gram of
// the workgroup's 128 bank states over the first kCrossFirst ordered
// candidates (4 waves x 32 states as row items, one 64-candidate chunk per
// column stage, a ring of stage buffers) stores each chunk sum as the chunk-sum Gram
// does, and every state whose running prefix reaches its bound within a chunk
// takes its first crossing there from the same weights, summed in candidate
// order (the two half-waves exchange their 4-candidate group sums); states that
// do not cross within the first part get R + 1, states already at their bound
// 0.  The bank's crossings found are added to ws.crossed.
template <int D, int P, bool FOLD, bool KV>
__global__ __launch_bounds__(64 * kWaves, D <= 128 ? 3 : 2) void k_first_part_mfma(dkv_bank bank, Geom g, Prm p,
                                                                                 Workspace ws, int32_t *out_first) {
  static_assert(kCkStride == 2 * kCT, "two 32-candidate tiles per chunk");
  const int b = blockIdx.y;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, n = l & 31, hw = l >> 5;
  const int m = ws.m[b], R = ws.R[b];
  if ((int)blockIdx.x * 32 * kWaves >= m) return;  // whole workgroup (the stages have barriers)
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  const int v = blockIdx.x * 32 * kWaves + wave * 32 + n;
  const bool rv = v < m;
  const int64_t row = (int64_t)(rb + min(v, m - 1));
  // the bound: the state violates once rho + P reaches ceil(T b / 2^k)
  const int64_t lim = ((int64_t)p.tau_num * bank.base[row] + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
  const int64_t thr = lim - bank.rho[row];
  const int nch = min((R + kCkStride - 1) / kCkStride, kCrossFirst / kCkStride);
  int first = thr > 0 ? R + 1 : 0;
  bool open = thr > 0;  // not yet crossed
  if (nch > 0) {
    RowFrag<D> rf;
    load_row_frag<D, FOLD, KV>(rf, Desc{static_cast<const uint16_t *>(bank.k), static_cast<const uint16_t *>(bank.v)},
                               row, bank.knorm[row], rv, -2.0f * p.inv_sigma2, p.inv_sigma2);
    int aoff[TileCfg<D>::kSteps];
    frag_offsets<D>(aoff);
    constexpr int KB = SCfg<D>::KEYB, AB = SCfg<D>::AUGB;
    // a ring of three stage buffers (two chunks in flight), two at descriptor
    // dimension 256, where three would leave one workgroup per CU
    constexpr int NBUF = D <= 128 ? 3 : 2;
    __shared__ __attribute__((aligned(1024))) char kbuf[NBUF][KB];
    __shared__ __attribute__((aligned(16))) char abuf[NBUF][AB];
    const StageOff<D> soff = stage_offsets<D>();
    auto issue = [&](int c, int buf) __attribute__((always_inline)) {
      stage_dma_seq<D, false>(soff, c * kCkStride, ws.sk, ws.saug, nullptr, kbuf[buf], abuf[buf], nullptr, (int64_t)nb,
                              g.N);
    };
    constexpr int kOps = stage_ops<D, false>();
    uint64_t run = 0;  // the state's prefix sum before chunk c
    for (int j = 0; j < NBUF - 1 && j < nch; ++j) issue(j, j);
    for (int c = 0; c < nch; ++c) {
      const int buf = c % NBUF;
      if (NBUF == 3 && c + 1 < nch) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kOps));  // chunk c + 1 stays in flight
      else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
      stage_barrier();  // every wave's loads of chunk c landed; every wave is done with chunk c - 1's buffer
      if (c + NBUF - 1 < nch) issue(c + NBUF - 1, (c + NBUF - 1) % NBUF);
      const f32x16 x0 = tile_mfma<D>(kbuf[buf], abuf[buf], 0, rf, aoff);
      const f32x16 x1 = tile_mfma<D>(kbuf[buf], abuf[buf], 1, rf, aoff);
      // weights in candidate order inside the lane: tile tl, register 4 k + j is
      // candidate 32 tl + 8 k + 4 hw + j of the chunk; candidates past R weigh nothing
      const int nvalid = min(kCkStride, R - c * kCkStride);
      uint32_t w[2][16], gsum[2][4];
#pragma unroll
      for (int tl = 0; tl < 2; ++tl) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          gsum[tl][k] = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            uint32_t W = weight_raw<P, FOLD>(tl ? x1[4 * k + j] : x0[4 * k + j], 8388608.0f) - kMagic;
            asm volatile("" : "+v"(W));  // computed for every lane, then masked
            W = 32 * tl + 8 * k + 4 * hw + j < nvalid ? W : 0u;
            w[tl][4 * k + j] = W;
            gsum[tl][k] += W;
          }
        }
      }
      uint32_t lane_tot = 0;
#pragma unroll
      for (int tl = 0; tl < 2; ++tl)
#pragma unroll
        for (int k = 0; k < 4; ++k) lane_tot += gsum[tl][k];
      const uint32_t tot = lane_tot + __shfl_xor(lane_tot, 32, 64);  // the chunk sum (at most 2^29)
      if (rv && hw == 0) ws.ck[(rb + v) * ws.nck + c] = tot;
      const bool hit = open && (int64_t)(run + tot) >= thr;
      if (__ballot(hit)) {  // uniform over the wave
        // inclusive prefixes in candidate order; the crossing is one plus the
        // number of candidates whose prefix is still below the need
        const uint32_t nd1 = hit ? (uint32_t)(thr - (int64_t)run) - 1u : 0u;
        uint32_t pr = 0, cnt = 0;
#pragma unroll
        for (int tl = 0; tl < 2; ++tl) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const uint32_t other = __shfl_xor(gsum[tl][k], 32, 64);
            uint32_t q = pr + (hw ? other : 0u);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              q += w[tl][4 * k + j];
              cnt += q <= nd1 ? 1u : 0u;
            }
            pr += gsum[tl][k] + other;
          }
        }
        cnt += __shfl_xor(cnt, 32, 64);
        if (hit) {
          first = c * kCkStride + (int)cnt + 1;
          open = false;
        }
      }
      run += tot;
    }
  }
  if (hw == 0 && rv) {
    ws.first[rb + v] = first;
    if (out_first) out_first[rb + v] = first;
  }
  const unsigned long long found = __ballot(hw == 0 && rv && first <= R);
  if (l == 0 && found) atomicAdd(&ws.crossed[b], (int)__popcll(found));
}

// Whether a group's crossing search must go on past its first part, the first
// L = kCrossFirst ordered candidates (every crossing r <= L found there).  c_r only grows with r and the evictions a bank can make at a tested
// length, max(0, m + r - M), are at most max(0, m + R - M); a bank with more
// crossings than that within the first part is infeasible at every r >= L
// (Eqs. 9-10), so r* < L for its group (Eq. 11), and the crossings within the
// first part decide r*, the mandatory releases (first crossing <= r*) and the
// projected densities at r* (chunks before r* only).  force: every state's
// first crossing is wanted.
__global__ __launch_bounds__(256) void k_cross_plan(Geom g, Workspace ws, int force) {
  const int grp = blockIdx.x * 256 + threadIdx.x;
  if (grp >= g.G) return;
  const int b0 = grp * g.gs, R = ws.R[b0];
  bool decided = R <= kCrossFirst;  // the first part tested every prefix
  for (int j = 0; j < g.gs && !decided; ++j) {
    const int b = b0 + j;
    decided = ws.crossed[b] > max(0, ws.m[b] + R - ws.M[b]);
  }
  ws.more[grp] = (!decided || (force && R > kCrossFirst)) ? 1 : 0;
}

// Chunk sums of the ordered prefixes [cfirst, clim) (splits of 1,024 from
// cfirst): the first part of the crossing search, or (second) the rest, for the
// groups whose first part left r* open.
template <int D, int P, bool FOLD, bool KV>
__global__ __launch_bounds__(64 * gram_waves<D>(), gram_waves<D>() == 4 ? 3 : 2) void k_chunk_part_mfma(
    dkv_bank bank, const void *seg_k, const void *seg_v, Geom g, Prm p, Workspace ws, int cfirst, int clim,
    int second) {
  if (second && !ws.more[blockIdx.z / g.gs]) return;
  constexpr int KB = SCfg<D>::KEYB, AB = SCfg<D>::AUGB;
  __shared__ __attribute__((aligned(1024))) char k0[KB], k1[KB], k2[KB];
  __shared__ __attribute__((aligned(16))) char a0[AB], a1[AB], a2[AB];
  const StageBufs<D> sb{k0, k1, k2, a0, a1, a2, nullptr};
  rowsum_body<D, P, RS_CHUNK, FOLD, KV>(bank, seg_k, seg_v, g, p, ws, nullptr, blockIdx.x, blockIdx.y, blockIdx.z, sb,
                                        cfirst, clim);
}

// Candidate keys and norms in score order, so that the ordered passes stream
// contiguous rows: one thread per 16-byte chunk of kGatherRows key rows
// (every load and store instruction covers whole rows).
constexpr int kGatherRows = 4;

// Positions [r0, r1) of the order (r1 <= N): the first part of the crossing
// search reads positions below kCrossFirst only, so the rest is copied (second)
// only for the groups whose first part left r* open.
template <int D, bool KV>
__global__ __launch_bounds__(256) void k_gather_sorted(const void *seg_k, const void *seg_v, Geom g, Workspace ws,
                                                       int r0, int r1, int second) {
  constexpr int CH = D / 8;      // 16-byte chunks per bf16 row
  constexpr int RPP = 256 / CH;  // rows per workgroup pass
  static_assert(kGatherRows <= CH, "one metadata lane per row of the group");
  const int b = blockIdx.y;
  const int c = threadIdx.x % CH;
  const int j0 = r0 + blockIdx.x * RPP * kGatherRows + threadIdx.x / CH;
  const size_t nb = (size_t)b * g.N;
  if (r0 + (int)blockIdx.x * RPP * kGatherRows >= r1) return;  // whole workgroup
  if (second && !ws.more[b / g.gs]) return;
  const Desc src{static_cast<const uint16_t *>(seg_k), static_cast<const uint16_t *>(seg_v)};
  // loads from clamped (in-range) rows, unconditional so that they overlap
  int xs[kGatherRows];
#pragma unroll
  for (int u = 0; u < kGatherRows; ++u) xs[u] = ws.order[nb + min(j0 + u * RPP, r1 - 1)];
  u32x4 tmp[kGatherRows];
#pragma unroll
  for (int u = 0; u < kGatherRows; ++u)
    tmp[u] = *reinterpret_cast<const u32x4 *>(desc_chunk<D, KV>(src, (int64_t)(nb + xs[u]), c));
#pragma unroll
  for (int u = 0; u < kGatherRows; ++u)
    if (j0 + u * RPP < r1) reinterpret_cast<u32x4 *>(ws.sk + (nb + j0 + u * RPP) * D)[c] = tmp[u];
  // lane c < kGatherRows of a row group copies the norm and norm step of row c
  if (c < kGatherRows) {
    const int j = j0 + c * RPP;
    if (j < r1) {
      const int x = ws.order[nb + j];
      ws.snorm[nb + j] = ws.cnorm[nb + x];
      ws.saug[nb + j] = ws.caug[nb + x];
    }
  }
}

// Score entry point outputs from the accumulated sums.
__global__ void k_score_out(Geom g, Workspace ws, int64_t *out_q, float *out_f) {
  const int b = blockIdx.y, x = blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= g.N) return;
  const size_t o = (size_t)b * g.N + x;
  const int m = ws.m[b];
  const int64_t A = ws.acol[o];
  if (out_q) out_q[o] = A;
  if (out_f) out_f[o] = m > 0 ? (float)(ldexp((double)A, ws.E[b] - 23) / (double)m) : 0.0f;
}

__global__ void k_density_out(Geom g, Workspace ws, int64_t *out) {
  const int b = blockIdx.y, i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= ws.m[b]) return;
  out[(size_t)b * g.Mcap + i] = ws.sub[(size_t)b * g.Mcap + i];
}

inline unsigned cdiv(int a, int b) { return (unsigned)((a + b - 1) / b); }

// D is the descriptor dimension: the key dimension, or twice it for the
// [K; V] geometry (KV: the candidates' values seg_v and bank.v are read too).
template <int D, int P, bool F, bool KV>
void mfma_update_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                      const dkv_update_out &out, const Workspace &ws, hipStream_t s, int stage) {
  constexpr int W = gram_waves<D>();
  const int T = 64 * W;
  const unsigned rowsM = cdiv(g.Mcap, 32 * W), rowsN = cdiv(g.N > 0 ? g.N : 1, 32 * W);
  const void *sv = seg.v;
  switch (stage) {
    case 0:  // score; the ordered copy is launched after the sort (stage 4)
      k_score_mfma<D, P, F, KV><<<rowsN * cdiv(g.Mcap, kColsPerSplit) * (unsigned)g.B, T, 0, s>>>(bank, seg.k, sv, g,
                                                                                                   p, ws);
      break;
    case 4: {  // the positions the first part of the crossing search reads
      const int r1 = min(g.N, kCrossFirst);
      k_gather_sorted<D, KV><<<dim3(cdiv(r1, 256 / (D / 8) * kGatherRows), g.B), 256, 0, s>>>(seg.k, sv, g, ws, 0, r1,
                                                                                             0);
      break;
    }
    case 1: {
      // The crossing search in two parts: the chunk sums of the first
      // kCrossFirst ordered candidates and the crossings within them; then, for
      // the groups that this leaves open (k_cross_plan), the chunk sums of the
      // rest and the whole search again.
      const dim3 xgrid(cdiv(g.Mcap, kWaves * kCrossWaveStates), g.B);
      k_first_part_mfma<D, P, F, KV><<<dim3(cdiv(g.Mcap, 32 * kWaves), g.B), 64 * kWaves, 0, s>>>(bank, g, p, ws,
                                                                                                out.first_cross);
      if (g.N > kCrossFirst) {
        k_cross_plan<<<cdiv(g.G, 256), 256, 0, s>>>(g, ws, out.first_cross != nullptr ? 1 : 0);
        k_gather_sorted<D, KV><<<dim3(cdiv(g.N - kCrossFirst, 256 / (D / 8) * kGatherRows), g.B), 256, 0, s>>>(
            seg.k, sv, g, ws, kCrossFirst, g.N, 1);
        k_chunk_part_mfma<D, P, F, KV><<<dim3(rowsM, cdiv(g.N - kCrossFirst, kChunksPerSplit * kCkStride), g.B), T,
                                         0, s>>>(bank, seg.k, sv, g, p, ws, kCrossFirst, 1 << 30, 1);
        k_cross_mfma<D, P, F, KV><<<xgrid, 64 * kWaves, 0, s>>>(bank, g, p, ws, out.first_cross);
      }
      break;
    }
    case 2:
      k_rowsum_mfma<D, P, RS_FIXUP, F, KV><<<dim3(rowsM, 1, g.B), T, 0, s>>>(bank, seg.k, sv, g, p, ws, out.rho_tilde);
      break;
    case 3: {
      // the work items, then a grid of at most kMaintWgs workgroups over them
      // (evicted states <= admitted <= N: at most rowsM x splits of N, plus
      // rowsN x (splits of Mcap + half splits of N) items per bank)
      k_maint_plan<<<1, kPlanThreads, 0, s>>>(g, ws, 32 * W);
      const unsigned y_ev = cdiv(g.N > 0 ? g.N : 1, kColsPerSplit), y_surv = cdiv(g.Mcap, kColsPerSplit);
      const unsigned long long bound =
          (unsigned long long)(rowsM * y_ev + (g.N > 0 ? rowsN : 0u) * (y_surv + 2 * y_ev)) * (unsigned)g.B;
      const unsigned nwg = (unsigned)(bound < kMaintWgs ? (bound > 0 ? bound : 1) : kMaintWgs);
      k_maint_mfma<D, P, F, KV><<<nwg, T, 0, s>>>(bank, seg.k, sv, g, p, ws);
      break;
    }
    default:
      break;
  }
}

// The +1 of t = 1 + u rides in the MFMA when sigma^2 <= 2^11 (exact there).
inline bool fold_one(const Prm &p) { return p.inv_sigma2 >= 1.0f / 2048.0f; }

template <int D, bool KV>
void mfma_stage_d(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                  const dkv_update_out &out, const Workspace &ws, hipStream_t s, int stage) {
  const bool f = fold_one(p);
  if (p.p == 1) f ? mfma_update_impl<D, 1, true, KV>(bank, seg, g, p, out, ws, s, stage) : mfma_update_impl<D, 1, false, KV>(bank, seg, g, p, out, ws, s, stage);
  else if (p.p == 2) f ? mfma_update_impl<D, 2, true, KV>(bank, seg, g, p, out, ws, s, stage) : mfma_update_impl<D, 2, false, KV>(bank, seg, g, p, out, ws, s, stage);
  else f ? mfma_update_impl<D, 4, true, KV>(bank, seg, g, p, out, ws, s, stage) : mfma_update_impl<D, 4, false, KV>(bank, seg, g, p, out, ws, s, stage);
}

template <int D, int P, bool F, bool KV>
void mfma_score_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                     int64_t *score_q, float *score_f, int64_t *density, const Workspace &ws, hipStream_t s) {
  constexpr int W = gram_waves<D>();
  const int T = 64 * W;
  if (g.N > 0 && (score_q || score_f)) {
    k_score_mfma<D, P, F, KV><<<cdiv(g.N, 32 * W) * cdiv(g.Mcap, kColsPerSplit) * (unsigned)g.B, T, 0, s>>>(
        bank, seg.k, seg.v, g, p, ws);
    k_score_out<<<dim3(cdiv(g.N, 256), g.B), 256, 0, s>>>(g, ws, score_q, score_f);
  }
  if (density) {
    k_rowsum_mfma<D, P, RS_DENSITY, F, KV><<<dim3(cdiv(g.Mcap, 32 * W), cdiv(g.Mcap, kColsPerSplit), g.B), T, 0,
                                              s>>>(bank, seg.k, seg.v, g, p, ws, density);
    k_density_out<<<dim3(cdiv(g.Mcap, 256), g.B), 256, 0, s>>>(g, ws, density);
  }
}

template <int D, bool KV>
void mfma_score_d(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p, int64_t *score_q,
                  float *score_f, int64_t *density, const Workspace &ws, hipStream_t s) {
  const bool f = fold_one(p);
  if (p.p == 1) f ? mfma_score_impl<D, 1, true, KV>(bank, seg, g, p, score_q, score_f, density, ws, s) : mfma_score_impl<D, 1, false, KV>(bank, seg, g, p, score_q, score_f, density, ws, s);
  else if (p.p == 2) f ? mfma_score_impl<D, 2, true, KV>(bank, seg, g, p, score_q, score_f, density, ws, s) : mfma_score_impl<D, 2, false, KV>(bank, seg, g, p, score_q, score_f, density, ws, s);
  else f ? mfma_score_impl<D, 4, true, KV>(bank, seg, g, p, score_q, score_f, density, ws, s) : mfma_score_impl<D, 4, false, KV>(bank, seg, g, p, score_q, score_f, density, ws, s);
}

inline bool kv_geometry(const Prm &p) { return (p.flags & DKV_POLICY_KV_DESCRIPTOR) != 0; }

}  // namespace

// Stage launchers used by the update sequence for bf16 banks:
// 0 score, 4 ordered copy, 1 crossing, 2 r* fix-up, 3 maintenance.  The
// descriptor dimension is the key dimension, or twice it for [K; V].
void launch_gram_mfma(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                      const dkv_update_out &out, const Workspace &ws, hipStream_t s, int stage) {
  if (kv_geometry(p)) {
    if (g.d == 128) mfma_stage_d<256, true>(bank, seg, g, p, out, ws, s, stage);
    else mfma_stage_d<128, true>(bank, seg, g, p, out, ws, s, stage);
  } else {
    if (g.d == 128) mfma_stage_d<128, false>(bank, seg, g, p, out, ws, s, stage);
    else mfma_stage_d<64, false>(bank, seg, g, p, out, ws, s, stage);
  }
}

void launch_score_mfma(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                       int64_t *score_q, float *score_f, int64_t *density, const Workspace &ws, hipStream_t s) {
  if (kv_geometry(p)) {
    if (g.d == 128) mfma_score_d<256, true>(bank, seg, g, p, score_q, score_f, density, ws, s);
    else mfma_score_d<128, true>(bank, seg, g, p, score_q, score_f, density, ws, s);
  } else {
    if (g.d == 128) mfma_score_d<128, false>(bank, seg, g, p, score_q, score_f, density, ws, s);
    else mfma_score_d<64, false>(bank, seg, g, p, score_q, score_f, density, ws, s);
  }
}

}  // namespace dkv
