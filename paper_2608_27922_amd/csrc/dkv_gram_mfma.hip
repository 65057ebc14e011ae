// Key-key Gram stages of the DensityKV update on bf16 MFMA (gfx950).
//
// Every Gram stage evaluates Soft-Riesz weights w(k_i, k_j) (Eq. 2) for a set
// of "row" items against a stream of "column" items and reduces them per row:
//
//   k_score_mfma   rows = candidates, columns = bank states:
//                  S_x = sum_i RNE(w_ix bs_i), Wcol_x = sum_i W_ix  (Eq. 6)
//   k_rowsum_mfma  row sums: per-64-candidate chunk sums over the ordered
//                  candidates (the prefix checkpoints of Eqs. 8-9), the r*
//                  fix-up, the exact maintenance (Supp. C) and the
//                  from-scratch bank density (Eq. 3)
//   k_cross_find   per bank state: the chunk in which its prefix density first
//                  reaches tau b, then the exact prefix length inside it
//
// The column range of every Gram is split over workgroups (grid dimension y);
// partial integer sums are combined with 64-bit atomic adds, which are exact
// and order-independent.
//
// Layout: a workgroup of 4 waves owns 128 row items; wave w owns 32 of them,
// held for the whole kernel as the B operand of v_mfma_f32_32x32x16_bf16
// (lane l <-> row item l % 32).  Column items stream through LDS in tiles of 32
// (double-buffered, padded rows) and form the A operand, so each lane ends up
// with 16 weights of its own row item and reduces them in registers.
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

constexpr int kWaves = 4;
constexpr int kRowsPerWG = 32 * kWaves;
constexpr int kCT = 32;  // column items per MFMA tile
constexpr int kSI = 64;  // column items per LDS stage (two tiles, two independent MFMA chains)

template <int D>
struct TileCfg {
  static constexpr int kSteps = D / 16;     // K steps over the key
  static constexpr int kStride = D + 24;    // bf16 per LDS row: key, 16 aug, 8 pad (odd multiple of 16 B)
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
  const float y = __builtin_amdgcn_rcpf(tp);
  const float e = __builtin_fmaf(-tp, y, 1.0f);
  const float w = __builtin_fmaf(e, y, y);
  return __float_as_uint(__builtin_fmaf(w, scale, 8388608.0f));
}

// Row fragment: B operand of every K step for this lane's row item.
template <int D>
struct RowFrag {
  bf16x8 b[TileCfg<D>::kSteps + 1];
};

// Load the B operand for row item (lane % 32): keys scaled by -2/sigma^2, then
// the aug step [1, 1, 1, n_hi, n_mid, n_lo, fold, 0] (half 0) / zeros (half 1).
template <int D, bool FOLD>
__device__ __forceinline__ void load_row_frag(RowFrag<D> &rf, const uint16_t *key, float norm, bool valid,
                                              float neg2_inv_s2, float inv_s2) {
  const int h = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int kk = 0; kk < TileCfg<D>::kSteps; ++kk) {
    u32x4 raw = {0, 0, 0, 0};
    if (valid) raw = *reinterpret_cast<const u32x4 *>(key + 16 * kk + 8 * h);
    u32x4 sc;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float lo = bf16_bits_to_f32((uint16_t)(raw[q] & 0xFFFF)) * neg2_inv_s2;
      const float hi = bf16_bits_to_f32((uint16_t)(raw[q] >> 16)) * neg2_inv_s2;
      sc[q] = (uint32_t)bf16_rne_bits(lo) | ((uint32_t)bf16_rne_bits(hi) << 16);
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

// Column stage staging: each of the 256 threads moves 16-byte chunks of the
// stage's keys; 64 threads write the aug columns.
template <int D>
struct ColStage {
  u32x4 chunk[(kSI * TileCfg<D>::kChunks) / (64 * kWaves)];
  u32x4 aug0;
};

// item_row(i) returns the element offset of column item i's key, or -1.
template <int D, class RowOf, class NormOf>
__device__ __forceinline__ void stage_load(ColStage<D> &st, const uint16_t *base, int j0, int ncols,
                                           RowOf row_of, NormOf norm_of, float inv_s2) {
  constexpr int kPer = (kSI * TileCfg<D>::kChunks) / (64 * kWaves);
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int c = threadIdx.x + q * 64 * kWaves;
    const int item = c / TileCfg<D>::kChunks, ch = c % TileCfg<D>::kChunks;
    u32x4 v = {0, 0, 0, 0};
    if (j0 + item < ncols) {
      const int64_t r = row_of(j0 + item);
      v = *reinterpret_cast<const u32x4 *>(base + r * D + ch * 8);
    }
    st.chunk[q] = v;
  }
  if (threadIdx.x < kSI) {
    u32x4 a = {0, 0, 0, 0};
    if (j0 + (int)threadIdx.x < ncols) {
      uint16_t nh, nm, nl;
      split3(norm_of(j0 + (int)threadIdx.x) * inv_s2, nh, nm, nl);
      a[0] = (uint32_t)nh | ((uint32_t)nm << 16);
      a[1] = (uint32_t)nl | ((uint32_t)kOne << 16);
      a[2] = (uint32_t)kOne | ((uint32_t)kOne << 16);
      a[3] = (uint32_t)kOne;  // times the row's fold slot
    }
    st.aug0 = a;
  }
}

template <int D>
__device__ __forceinline__ void stage_store(const ColStage<D> &st, uint16_t *lds) {
  constexpr int kPer = (kSI * TileCfg<D>::kChunks) / (64 * kWaves);
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int c = threadIdx.x + q * 64 * kWaves;
    const int item = c / TileCfg<D>::kChunks, ch = c % TileCfg<D>::kChunks;
    *reinterpret_cast<u32x4 *>(lds + item * TileCfg<D>::kStride + ch * 8) = st.chunk[q];
  }
  if (threadIdx.x < kSI) {
    *reinterpret_cast<u32x4 *>(lds + threadIdx.x * TileCfg<D>::kStride + D) = st.aug0;
    *reinterpret_cast<u32x4 *>(lds + threadIdx.x * TileCfg<D>::kStride + D + 8) = u32x4{0, 0, 0, 0};
  }
}

// u for the 16 (column item, row item) pairs of this lane: column items
// m_i = 8 (i / 4) + 4 h + (i % 4), row item = lane % 32.
template <int D>
__device__ __forceinline__ f32x16 tile_u(const uint16_t *lds, const RowFrag<D> &rf) {
  const int l = threadIdx.x & 63;
  const uint16_t *src = lds + (l & 31) * TileCfg<D>::kStride + 8 * (l >> 5);
  bf16x8 a[TileCfg<D>::kSteps + 1];
#pragma unroll
  for (int kk = 0; kk <= TileCfg<D>::kSteps; ++kk)
    a[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(src + 16 * kk));
  f32x16 acc = {};
#pragma unroll
  for (int kk = 0; kk <= TileCfg<D>::kSteps; ++kk)
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk], rf.b[kk], acc, 0, 0, 0);
  return acc;
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

template <int D, int P, bool FOLD>
__global__ __launch_bounds__(64 * kWaves, 2) void k_score_mfma(dkv_bank bank, const void *seg_k, Geom g, Prm p,
                                                           Workspace ws) {
  const int b = blockIdx.z;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const int x = blockIdx.x * kRowsPerWG + wave * 32 + n;
  const int m = ws.m[b];
  const int c0 = blockIdx.y * kColsPerSplit;
  if (c0 >= m) return;
  const int ncols = min(kColsPerSplit, m - c0);
  __shared__ __attribute__((aligned(16))) uint16_t tile[2][kSI * TileCfg<D>::kStride];
  __shared__ __attribute__((aligned(16))) float tbs[2][kSI];
  const uint16_t *K = static_cast<const uint16_t *>(seg_k);
  const uint16_t *BK = static_cast<const uint16_t *>(bank.k);
  const bool rv = x < g.N;
  const size_t xr = (size_t)b * g.N + (rv ? x : 0);
  RowFrag<D> rf;
  load_row_frag<D, FOLD>(rf, K + xr * D, rv ? ws.cnorm[xr] : 0.0f, rv, -2.0f * p.inv_sigma2, p.inv_sigma2);
  const size_t rb = (size_t)b * g.Mcap + c0;
  auto row_of = [&](int i) -> int64_t { return (int64_t)(rb + i); };
  auto norm_of = [&](int i) -> float { return bank.knorm[rb + i]; };
  uint64_t A64 = 0, W64 = 0;
  const int ns = (ncols + kSI - 1) / kSI;
  ColStage<D> st;
  float bs_next = 0.0f;
  stage_load<D>(st, BK, 0, ncols, row_of, norm_of, p.inv_sigma2);
  if (threadIdx.x < kSI) bs_next = (int)threadIdx.x < ncols ? ws.bs[rb + threadIdx.x] : 0.0f;
  stage_store<D>(st, tile[0]);
  if (threadIdx.x < kSI) tbs[0][threadIdx.x] = bs_next;
  __syncthreads();
  // epilogue of one 32-column tile: integer sums of W and of the scaled score terms
  auto epi = [&](auto mask_tag, const f32x16 &u, const float *tb, int nvalid, uint32_t &sw, uint32_t &sa) {
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
    sw = 0;
    sa = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float tt = FOLD ? u[i] : 1.0f + u[i];
      float tp = tt;
      if constexpr (P >= 2) tp = tt * tt;
      if constexpr (P == 4) tp = tp * tp;
      const float y = __builtin_amdgcn_rcpf(tp);
      const float e = __builtin_fmaf(-tp, y, 1.0f);
      const float w = __builtin_fmaf(e, y, y);
      uint32_t rw = __float_as_uint(__builtin_fmaf(w, 8388608.0f, 8388608.0f));
      uint32_t ra = __float_as_uint(__builtin_fmaf(w, bsv[i], 8388608.0f));
      if constexpr (MASK) {
        const bool ok = col_of_reg(i, h) < nvalid;
        rw = ok ? rw : kMagic;
        ra = ok ? ra : kMagic;
      }
      sw += rw;
      sa += ra;
    }
    sw -= 16u * kMagic;
    sa -= 16u * kMagic;
  };
  using Full = std::integral_constant<bool, false>;
  using Part = std::integral_constant<bool, true>;
  for (int t = 0; t < ns; ++t) {
    const int cur = t & 1;
    const int j0n = (t + 1) * kSI;
    if (t + 1 < ns) {
      stage_load<D>(st, BK, j0n, ncols, row_of, norm_of, p.inv_sigma2);
      if (threadIdx.x < kSI) bs_next = j0n + (int)threadIdx.x < ncols ? ws.bs[rb + j0n + threadIdx.x] : 0.0f;
    }
    const int nv0 = ncols - t * kSI;
    const f32x16 u0 = tile_u<D>(tile[cur], rf);
    const f32x16 u1 = tile_u<D>(tile[cur] + kCT * TileCfg<D>::kStride, rf);
    uint32_t sw, sa;
    if (nv0 >= kSI) {
      epi(Full{}, u0, tbs[cur], kCT, sw, sa);
      W64 += sw;
      A64 += sa;
      epi(Full{}, u1, tbs[cur] + kCT, kCT, sw, sa);
      W64 += sw;
      A64 += sa;
    } else {
      epi(Part{}, u0, tbs[cur], nv0, sw, sa);
      W64 += sw;
      A64 += sa;
      if (nv0 > kCT) {
        epi(Part{}, u1, tbs[cur] + kCT, nv0 - kCT, sw, sa);
        W64 += sw;
        A64 += sa;
      }
    }
    if (t + 1 < ns) {
      stage_store<D>(st, tile[cur ^ 1]);
      if (threadIdx.x < kSI) tbs[cur ^ 1][threadIdx.x] = bs_next;
    }
    __syncthreads();
  }
  const uint64_t Wt = W64 + __shfl_xor(W64, 32, 64);
  const uint64_t At = A64 + __shfl_xor(A64, 32, 64);
  if (!rv || h != 0) return;
  const size_t o = (size_t)b * g.N + x;
  atomicAdd(reinterpret_cast<unsigned long long *>(&ws.acol[o]), (unsigned long long)At);
  atomicAdd(reinterpret_cast<unsigned long long *>(&ws.wcol[o]), (unsigned long long)Wt);
}

// ---------------------------------------------------------------------------
// Row sums.  MODE selects rows, columns and where the sum goes.
// ---------------------------------------------------------------------------
enum RowSumMode { RS_CHUNK = 0, RS_FIXUP = 1, RS_SURV_EV = 2, RS_ADM_BASE = 3, RS_ADM_MUT = 4, RS_DENSITY = 5 };

constexpr int kChunksPerSplit = 1024 / kCkStride;   // RS_CHUNK: 1024 ordered candidates per workgroup

template <int D, int P, int MODE, bool FOLD>
__global__ __launch_bounds__(64 * kWaves, 3) void k_rowsum_mfma(dkv_bank bank, const void *seg_k, Geom g, Prm p,
                                                            Workspace ws, int64_t *out) {
  const int b = blockIdx.z;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  const int m = ws.m[b];
  const uint16_t *SK = static_cast<const uint16_t *>(seg_k);
  const uint16_t *BK = static_cast<const uint16_t *>(bank.k);
  const uint16_t *SORTK = ws.sk;
  constexpr bool kNeedEv = MODE == RS_SURV_EV || MODE == RS_ADM_BASE || MODE == RS_ADM_MUT;
  const int n_ev = kNeedEv ? ws.n_ev[b] : 0;
  const int rs = (MODE == RS_FIXUP || kNeedEv) ? ws.r_star[b / g.gs] : 0;
  const int n_surv = m - n_ev;
  const bool adm_by_ev = n_ev <= n_surv;
  // rows
  int nrows;
  if constexpr (MODE == RS_CHUNK || MODE == RS_FIXUP || MODE == RS_DENSITY) nrows = m;
  else if constexpr (MODE == RS_SURV_EV) nrows = n_surv;
  else nrows = rs;
  if ((int)blockIdx.x * kRowsPerWG >= nrows) return;
  // columns of this workgroup: [c0, c1) of the mode's column list
  int c0 = 0, c1 = 0;
  if constexpr (MODE == RS_CHUNK) {
    const int R = ws.R[b];
    c0 = blockIdx.y * kChunksPerSplit * kCkStride;
    c1 = min(R, c0 + kChunksPerSplit * kCkStride);
  } else if constexpr (MODE == RS_FIXUP) {
    c0 = (rs / kCkStride) * kCkStride;
    c1 = rs;
  } else {
    int total;
    if constexpr (MODE == RS_SURV_EV) total = n_ev;
    else if constexpr (MODE == RS_ADM_BASE) total = adm_by_ev ? n_ev : n_surv;
    else if constexpr (MODE == RS_ADM_MUT) total = rs;
    else total = m;
    c0 = blockIdx.y * kColsPerSplit;
    c1 = min(total, c0 + kColsPerSplit);
  }
  if (MODE != RS_FIXUP && c0 >= c1) return;  // the fix-up always writes rho~, even for r* % 256 == 0
  const int v = blockIdx.x * kRowsPerWG + wave * 32 + n;
  const bool rv = v < nrows;
  // row item
  const uint16_t *rkey = BK + rb * D;
  float rnorm = 0.0f;
  size_t out_idx = 0;
  if (rv) {
    if constexpr (MODE == RS_CHUNK || MODE == RS_FIXUP || MODE == RS_DENSITY) {
      rkey = BK + (rb + v) * D;
      rnorm = bank.knorm[rb + v];
      out_idx = rb + v;
    } else if constexpr (MODE == RS_SURV_EV) {
      const int s = ws.surv_list[rb + v];
      rkey = BK + (rb + s) * D;
      rnorm = bank.knorm[rb + s];
      out_idx = rb + s;
    } else {
      const int x = ws.adm_list[nb + v];
      rkey = SK + (nb + x) * D;
      rnorm = ws.cnorm[nb + x];
      out_idx = nb + v;
    }
  }
  RowFrag<D> rf;
  load_row_frag<D, FOLD>(rf, rkey, rnorm, rv, -2.0f * p.inv_sigma2, p.inv_sigma2);
  // column items (absolute index j in the mode's list)
  auto row_of = [&](int j) -> int64_t {
    if constexpr (MODE == RS_CHUNK || MODE == RS_FIXUP) return (int64_t)(nb + j);
    else if constexpr (MODE == RS_SURV_EV) return (int64_t)(rb + ws.ev_list[rb + j]);
    else if constexpr (MODE == RS_ADM_BASE)
      return (int64_t)(rb + (adm_by_ev ? ws.ev_list[rb + j] : ws.surv_list[rb + j]));
    else if constexpr (MODE == RS_ADM_MUT) return (int64_t)(nb + ws.adm_list[nb + j]);
    else return (int64_t)(rb + j);
  };
  auto norm_of = [&](int j) -> float {
    if constexpr (MODE == RS_CHUNK || MODE == RS_FIXUP) return ws.snorm[nb + j];
    else if constexpr (MODE == RS_SURV_EV) return bank.knorm[rb + ws.ev_list[rb + j]];
    else if constexpr (MODE == RS_ADM_BASE)
      return bank.knorm[rb + (adm_by_ev ? ws.ev_list[rb + j] : ws.surv_list[rb + j])];
    else if constexpr (MODE == RS_ADM_MUT) return ws.cnorm[nb + ws.adm_list[nb + j]];
    else return bank.knorm[rb + j];
  };
  const uint16_t *colbase = (MODE == RS_CHUNK || MODE == RS_FIXUP) ? SORTK : (MODE == RS_ADM_MUT ? SK : BK);
  constexpr bool kDiag = (MODE == RS_ADM_MUT || MODE == RS_DENSITY);
  __shared__ __attribute__((aligned(16))) uint16_t tile[2][kSI * TileCfg<D>::kStride];
  uint64_t S64 = 0;
  uint32_t chunk_sum = 0;
  const int ncols = c1 - c0;
  const int ns = (ncols + kSI - 1) / kSI;
  ColStage<D> st;
  auto row_of_rel = [&](int j) -> int64_t { return row_of(c0 + j); };
  auto norm_of_rel = [&](int j) -> float { return norm_of(c0 + j); };
  if (ns > 0) {
    stage_load<D>(st, colbase, 0, ncols, row_of_rel, norm_of_rel, p.inv_sigma2);
    stage_store<D>(st, tile[0]);
  }
  __syncthreads();
  const int wg_row0 = blockIdx.x * kRowsPerWG;
  // sum of the lane's 16 weights of one 32-column tile starting at list index j0
  auto tile_sum = [&](const f32x16 &u, int j0, int nvalid) -> uint32_t {
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
  for (int t = 0; t < ns; ++t) {
    const int cur = t & 1;
    if (t + 1 < ns) stage_load<D>(st, colbase, (t + 1) * kSI, ncols, row_of_rel, norm_of_rel, p.inv_sigma2);
    const f32x16 u0 = tile_u<D>(tile[cur], rf);
    const f32x16 u1 = tile_u<D>(tile[cur] + kCT * TileCfg<D>::kStride, rf);
    const int nv0 = ncols - t * kSI;
    const int j0 = c0 + t * kSI;
    uint32_t s2 = tile_sum(u0, j0, nv0);
    if (nv0 > kCT) s2 += tile_sum(u1, j0 + kCT, nv0 - kCT);
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
    if (t + 1 < ns) stage_store<D>(st, tile[cur ^ 1]);
    __syncthreads();
  }
  if constexpr (MODE == RS_CHUNK) return;
  uint64_t tot = S64;
  if constexpr (MODE == RS_FIXUP) {
    // plus the whole chunks before r*: the two half-waves sum alternate 4-chunk groups
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
  }
  tot += __shfl_xor(tot, 32, 64);
  if (!rv || h != 0) return;
  if constexpr (MODE == RS_FIXUP) {
    const size_t row = rb + v;
    const int64_t rt = bank.rho[row] + (int64_t)tot;
    ws.rho_t[row] = rt;
    if (out) out[row] = rt;
  } else {
    int64_t *dst = (MODE == RS_SURV_EV || MODE == RS_DENSITY) ? ws.sub : (MODE == RS_ADM_BASE ? ws.sub_adm : ws.mut_adm);
    atomicAdd(reinterpret_cast<unsigned long long *>(&dst[out_idx]), (unsigned long long)tot);
  }
}

// ---------------------------------------------------------------------------
// First violating prefix length of every bank state (Eqs. 8-9).
// k_cross_scan: thread per state; the first 64-candidate chunk whose sum
// lifts the prefix density to tau b.  States that never reach it get R + 1;
// the others are listed for k_cross_find, which re-walks that one chunk (one
// ordered candidate per lane, same binary32 weights) for the exact length.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_cross_scan(dkv_bank bank, Geom g, Prm p, Workspace ws, int32_t *out_first) {
  const int b = blockIdx.y, i = blockIdx.x * 256 + threadIdx.x;
  const int m = ws.m[b], R = ws.R[b];
  if (i >= m) return;
  const size_t rb = (size_t)b * g.Mcap, row = rb + i;
  const int64_t lim = ((int64_t)p.tau_num * bank.base[row] + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
  const int64_t thr = lim - bank.rho[row];
  int first = R + 1;
  if (thr <= 0) {
    first = 0;
  } else {
    const int nch = (R + kCkStride - 1) / kCkStride;
    const uint4 *ckr = reinterpret_cast<const uint4 *>(ws.ck + row * ws.nck);
    const int n4 = (nch + 3) / 4;
    int64_t P = 0;
    // batches of 8 x 4 chunk sums, all loads of a batch in flight together
    for (int c8 = 0; c8 < n4; c8 += 8) {
      uint4 q[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) q[e] = c8 + e < n4 ? ckr[c8 + e] : uint4{0, 0, 0, 0};
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const int c = 4 * c8 + e;
        const uint32_t v = e % 4 == 0 ? q[e / 4].x : e % 4 == 1 ? q[e / 4].y : e % 4 == 2 ? q[e / 4].z : q[e / 4].w;
        if (c >= nch) break;
        if (P + v >= thr) {
          const int k = atomicAdd(&ws.xcount[b], 1);
          ws.xlist[rb + k] = i | (c << 16);
          ws.xbefore[rb + k] = P;
          return;  // first written by k_cross_find
        }
        P += v;
      }
    }
  }
  ws.first[row] = first;
  if (out_first) out_first[row] = first;
}

template <int D, int P>
__global__ __launch_bounds__(256) void k_cross_find(dkv_bank bank, Geom g, Prm p, Workspace ws, int32_t *out_first) {
  const int b = blockIdx.y;
  const int l = threadIdx.x & 63;
  const int R = ws.R[b];
  const int cnt = ws.xcount[b];
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  {
    const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (k >= cnt) return;
    const int ent = ws.xlist[rb + k];
    const int i = ent & 0xFFFF, c = ent >> 16;
    const int64_t before = ws.xbefore[rb + k];
    const size_t row = rb + i;
    const int64_t lim = ((int64_t)p.tau_num * bank.base[row] + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
    const int64_t thr = lim - bank.rho[row];
    const uint16_t *rk = static_cast<const uint16_t *>(bank.k) + row * D;
    const float nr = bank.knorm[row];
    // one ordered candidate per lane: column c * 64 + l
    static_assert(kCkStride == 64, "one column per lane");
    const int col = c * kCkStride + l;
    uint32_t W = 0;
    if (col < R) {
      const uint16_t *ckey = ws.sk + (nb + col) * D;
      float acc = 0.0f;
#pragma unroll
      for (int j = 0; j < D; j += 8) {
        const u32x4 a = *reinterpret_cast<const u32x4 *>(rk + j);
        const u32x4 bb = *reinterpret_cast<const u32x4 *>(ckey + j);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc = __builtin_fmaf(__uint_as_float(a[e] << 16), __uint_as_float(bb[e] << 16), acc);
          acc = __builtin_fmaf(__uint_as_float(a[e] & 0xFFFF0000u), __uint_as_float(bb[e] & 0xFFFF0000u), acc);
        }
      }
      const float d2 = (nr + ws.snorm[nb + col]) - 2.0f * acc;
      W = weight_raw<P, false>(d2 * p.inv_sigma2, 8388608.0f) - kMagic;
    }
    uint32_t incl = W;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(incl, o, 64);
      if (l >= o) incl += y;
    }
    const unsigned long long hl = __ballot(before + (int64_t)incl >= thr);
    const int first = hl != 0 ? c * kCkStride + (__ffsll(hl) - 1) + 1
                              : min(R, (c + 1) * kCkStride);  // unreachable when both passes agree (exact Gram)
    if (l == 0) {
      ws.first[row] = first;
      if (out_first) out_first[row] = first;
    }
  }
}

// Candidate keys and norms in score order (contiguous rows for the ordered passes).
template <int D>
__global__ __launch_bounds__(256) void k_gather_sorted(const void *seg_k, Geom g, Workspace ws) {
  const int b = blockIdx.y;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6), l = threadIdx.x & 63;
  if (j >= g.N) return;
  const size_t nb = (size_t)b * g.N;
  const int x = ws.order[nb + j];
  const uint32_t *src = reinterpret_cast<const uint32_t *>(static_cast<const uint16_t *>(seg_k) + (nb + x) * D);
  uint32_t *dst = reinterpret_cast<uint32_t *>(ws.sk + (nb + j) * D);
  for (int e = l; e < D / 2; e += 64) dst[e] = src[e];
  if (l == 0) ws.snorm[nb + j] = ws.cnorm[nb + x];
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

template <int D, int P, bool F>
void mfma_update_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                      const dkv_update_out &out, const Workspace &ws, hipStream_t s, int stage) {
  const int T = 64 * kWaves;
  const unsigned rowsM = cdiv(g.Mcap, kRowsPerWG), rowsN = cdiv(g.N > 0 ? g.N : 1, kRowsPerWG);
  switch (stage) {
    case 0:  // score + sorted copy is launched after the sort (stage 4)
      k_score_mfma<D, P, F><<<dim3(rowsN, cdiv(g.Mcap, kColsPerSplit), g.B), T, 0, s>>>(bank, seg.k, g, p, ws);
      break;
    case 4:
      k_gather_sorted<D><<<dim3(cdiv(g.N, 4), g.B), 256, 0, s>>>(seg.k, g, ws);
      break;
    case 1: {
      if (g.N > 0)
        k_rowsum_mfma<D, P, RS_CHUNK, F><<<dim3(rowsM, cdiv(g.N, kChunksPerSplit * kCkStride), g.B), T, 0, s>>>(
            bank, seg.k, g, p, ws, nullptr);
      k_cross_scan<<<dim3(cdiv(g.Mcap, 256), g.B), 256, 0, s>>>(bank, g, p, ws, out.first_cross);
      k_cross_find<D, P><<<dim3(cdiv(g.Mcap, 4), g.B), 256, 0, s>>>(bank, g, p, ws, out.first_cross);
      break;
    }
    case 2:
      k_rowsum_mfma<D, P, RS_FIXUP, F><<<dim3(rowsM, 1, g.B), T, 0, s>>>(bank, seg.k, g, p, ws, out.rho_tilde);
      break;
    case 3:
      k_rowsum_mfma<D, P, RS_SURV_EV, F><<<dim3(rowsM, cdiv(g.Mcap, kColsPerSplit), g.B), T, 0, s>>>(bank, seg.k, g, p, ws, nullptr);
      if (g.N > 0) {
        k_rowsum_mfma<D, P, RS_ADM_BASE, F><<<dim3(rowsN, cdiv(g.Mcap, kColsPerSplit), g.B), T, 0, s>>>(bank, seg.k, g, p, ws, nullptr);
        k_rowsum_mfma<D, P, RS_ADM_MUT, F><<<dim3(rowsN, cdiv(g.N, kColsPerSplit), g.B), T, 0, s>>>(bank, seg.k, g, p, ws, nullptr);
      }
      break;
    default:
      break;
  }
}

// The +1 of t = 1 + u rides in the MFMA when sigma^2 <= 2^11 (exact there).
inline bool fold_one(const Prm &p) { return p.inv_sigma2 >= 1.0f / 2048.0f; }

template <int D>
void mfma_stage_d(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                  const dkv_update_out &out, const Workspace &ws, hipStream_t s, int stage) {
  const bool f = fold_one(p);
  if (p.p == 1) f ? mfma_update_impl<D, 1, true>(bank, seg, g, p, out, ws, s, stage) : mfma_update_impl<D, 1, false>(bank, seg, g, p, out, ws, s, stage);
  else if (p.p == 2) f ? mfma_update_impl<D, 2, true>(bank, seg, g, p, out, ws, s, stage) : mfma_update_impl<D, 2, false>(bank, seg, g, p, out, ws, s, stage);
  else f ? mfma_update_impl<D, 4, true>(bank, seg, g, p, out, ws, s, stage) : mfma_update_impl<D, 4, false>(bank, seg, g, p, out, ws, s, stage);
}

template <int D, int P, bool F>
void mfma_score_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                     int64_t *score_q, float *score_f, int64_t *density, const Workspace &ws, hipStream_t s) {
  const int T = 64 * kWaves;
  if (g.N > 0 && (score_q || score_f)) {
    k_score_mfma<D, P, F><<<dim3(cdiv(g.N, kRowsPerWG), cdiv(g.Mcap, kColsPerSplit), g.B), T, 0, s>>>(bank, seg.k, g, p, ws);
    k_score_out<<<dim3(cdiv(g.N, 256), g.B), 256, 0, s>>>(g, ws, score_q, score_f);
  }
  if (density) {
    k_rowsum_mfma<D, P, RS_DENSITY, F><<<dim3(cdiv(g.Mcap, kRowsPerWG), cdiv(g.Mcap, kColsPerSplit), g.B), T, 0, s>>>(
        bank, seg.k, g, p, ws, density);
    k_density_out<<<dim3(cdiv(g.Mcap, 256), g.B), 256, 0, s>>>(g, ws, density);
  }
}

}  // namespace

// Stage launchers used by the update sequence for bf16 banks:
// 0 score, 4 ordered copy, 1 crossing, 2 r* fix-up, 3 maintenance.
void launch_gram_mfma(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                      const dkv_update_out &out, const Workspace &ws, hipStream_t s, int stage) {
  if (g.d == 128) mfma_stage_d<128>(bank, seg, g, p, out, ws, s, stage);
  else mfma_stage_d<64>(bank, seg, g, p, out, ws, s, stage);
}

void launch_score_mfma(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                       int64_t *score_q, float *score_f, int64_t *density, const Workspace &ws, hipStream_t s) {
  auto go = [&](auto dtag, auto ptag) {
    constexpr int D = decltype(dtag)::value, P = decltype(ptag)::value;
    if (fold_one(p)) mfma_score_impl<D, P, true>(bank, seg, g, p, score_q, score_f, density, ws, s);
    else mfma_score_impl<D, P, false>(bank, seg, g, p, score_q, score_f, density, ws, s);
  };
  using I64 = std::integral_constant<int, 64>;
  using I128 = std::integral_constant<int, 128>;
  using P1 = std::integral_constant<int, 1>;
  using P2 = std::integral_constant<int, 2>;
  using P4 = std::integral_constant<int, 4>;
  if (g.d == 128) {
    if (p.p == 1) go(I128{}, P1{});
    else if (p.p == 2) go(I128{}, P2{});
    else go(I128{}, P4{});
  } else {
    if (p.p == 1) go(I64{}, P1{});
    else if (p.p == 2) go(I64{}, P2{});
    else go(I64{}, P4{});
  }
}

}  // namespace dkv
