// Native attention over [retained bank; local window] on gfx950.
//
// out = softmax(q K^T * scale) V with K = [bank k[0:m_b]; window k], the
// backbone's own attention reading the retained bank together with the local
// window (Sec. 1, Fig. 1; logit of Sec. 3.2).  Online (streaming) softmax in
// fp32 over key tiles staged in LDS; exp2 with the scale folded into log2(e).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "dkv_internal.hpp"

namespace dkv {
namespace {

constexpr int kAThreads = 256;
constexpr int kATile = 32;

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// One thread per query row; every thread of the block walks the same key tiles.
template <int D, int DT>
__global__ __launch_bounds__(kAThreads) void k_attn_rowwise(dkv_bank bank, const void *q, int nq,
                                                            const void *wk, const void *wv, int nw,
                                                            void *out, float scale_log2, Geom g) {
  const int b = blockIdx.y, qi = blockIdx.x * kAThreads + threadIdx.x;
  const bool act = qi < nq;
  const int M = clampi(bank.budget[b], 0, g.Mcap);
  const int m = clampi(bank.occupancy[b], 0, M);
  const int total = m + nw;
  __shared__ float tk[kATile][D];
  __shared__ float tv[kATile][D];
  float qr[D], o[D];
  const size_t qrow = (size_t)b * nq + qi;
  if (act) {
#pragma unroll
    for (int j = 0; j < D; ++j) qr[j] = load_elem<DT>(q, qrow * D + j);
  }
#pragma unroll
  for (int j = 0; j < D; ++j) o[j] = 0.0f;
  float mx = -INFINITY, l = 0.0f;
  for (int t0 = 0; t0 < total; t0 += kATile) {
    const int nc = min(kATile, total - t0);
    __syncthreads();
    for (int t = threadIdx.x; t < kATile * D; t += kAThreads) {
      const int c = t / D, j = t % D;
      const int key = t0 + c;
      float kv = 0.0f, vv = 0.0f;
      if (c < nc) {
        if (key < m) {
          const size_t r = ((size_t)b * g.Mcap + key) * D + j;
          kv = load_elem<DT>(bank.k, r);
          vv = load_elem<DT>(bank.v, r);
        } else {
          const size_t r = ((size_t)b * nw + (key - m)) * D + j;
          kv = load_elem<DT>(wk, r);
          vv = load_elem<DT>(wv, r);
        }
      }
      tk[c][j] = kv;
      tv[c][j] = vv;
    }
    __syncthreads();
    if (!act) continue;
    float s[kATile];
    float tmax = -INFINITY;
    for (int c = 0; c < nc; ++c) {
      float acc = 0.0f;
#pragma unroll
      for (int j = 0; j < D; ++j) acc = __builtin_fmaf(qr[j], tk[c][j], acc);
      s[c] = acc * scale_log2;
      tmax = fmaxf(tmax, s[c]);
    }
    const float mnew = fmaxf(mx, tmax);
    const float corr = exp2f(mx - mnew);
    l *= corr;
#pragma unroll
    for (int j = 0; j < D; ++j) o[j] *= corr;
    for (int c = 0; c < nc; ++c) {
      const float pr = exp2f(s[c] - mnew);
      l += pr;
#pragma unroll
      for (int j = 0; j < D; ++j) o[j] = __builtin_fmaf(pr, tv[c][j], o[j]);
    }
    mx = mnew;
  }
  if (!act) return;
  const float inv = l > 0.0f ? 1.0f / l : 0.0f;
  if constexpr (DT == DKV_BF16) {
    uint16_t *op = static_cast<uint16_t *>(out);
#pragma unroll
    for (int j = 0; j < D; ++j) op[qrow * D + j] = f32_to_bf16_bits(o[j] * inv);
  } else {
    float *op = static_cast<float *>(out);
#pragma unroll
    for (int j = 0; j < D; ++j) op[qrow * D + j] = o[j] * inv;
  }
}


// ---------------------------------------------------------------------------
// bf16 path on MFMA (v_mfma_f32_32x32x16_bf16).
//
// A workgroup of 4 waves owns 128 queries, 32 per wave.  Per tile of 64 keys:
//   S^T = K Q^T     A = K tile (LDS), B = Q^T (registers): lane l <-> query
//                   l % 32, registers <-> keys, so the softmax row statistics
//                   stay inside the lane (plus one exchange with lane l ^ 32);
//   O^T += V^T P^T  B = P straight from the S registers (bf16); A = V^T read
//                   from the row-major V tile with the transposing LDS read
//                   (ds_read_b64_tr_b16).  Inside each 16-key K step the key
//                   order is permuted identically in both operands
//                   (slot 8h + j <-> key 8 (j / 4) + 4 h + j % 4).
// K and V tiles go global -> LDS with 16-byte direct-to-LDS loads (no VGPR
// staging), double-buffered; rows are stored with an XOR swizzle of their
// 16-byte chunks so that both the K reads and the transposed V reads are free
// of LDS bank conflicts.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kFWaves = 4;
constexpr int kFQ = 32 * kFWaves;  // queries per workgroup
constexpr int kFK = 64;            // keys per tile

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

template <int D>
struct FCfg {
  static constexpr int kRowBytes = 2 * D;           // one K or V row
  static constexpr int kChunks = D / 8;             // 16-byte chunks per row
  static constexpr int kRowsPerLoad = 1024 / kRowBytes;   // rows per 1 KB direct load
  static constexpr int kLoadsPerTile = kFK / kRowsPerLoad;  // per tensor, per workgroup
  static constexpr int kTileBytes = kFK * kRowBytes;
};

// Physical 16-byte chunk of logical chunk c of row r (K: conflict-free 16-byte
// reads of one chunk across 16 rows; V: conflict-free transposed 8-byte reads
// of 4 chunks across 4 rows).
template <int D>
__device__ __forceinline__ int k_swz(int r, int c) { return c ^ (r % FCfg<D>::kChunks); }
template <int D>
__device__ __forceinline__ int v_swz(int r, int c) { return c ^ ((4 * (r % 4)) % FCfg<D>::kChunks); }

// Issue the direct-to-LDS loads of one tile (rows [0, nvalid) of kbase/vbase;
// rows beyond nvalid repeat the last real row so that every value is finite).
template <int D>
__device__ __forceinline__ void ftile_issue(const uint16_t *kbase, const uint16_t *vbase, int nvalid,
                                            char *kbuf, char *vbuf) {
  constexpr int RPL = FCfg<D>::kRowsPerLoad, CH = FCfg<D>::kChunks;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int rsub = l / CH, pc = l % CH;
#pragma unroll
  for (int q = 0; q < FCfg<D>::kLoadsPerTile / kFWaves; ++q) {
    const int blk = wave * (FCfg<D>::kLoadsPerTile / kFWaves) + q;
    const int r = blk * RPL + rsub;
    const int rr = r < nvalid ? r : nvalid - 1;
    __builtin_amdgcn_global_load_lds(kbase + (size_t)rr * D + 8 * k_swz<D>(r, pc),
                                     (lds_void *)(kbuf + blk * 1024), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(vbase + (size_t)rr * D + 8 * v_swz<D>(r, pc),
                                     (lds_void *)(vbuf + blk * 1024), 16, 0, 0);
  }
}

template <int D>
__global__ __launch_bounds__(64 * kFWaves, 2) void k_attn_mfma(dkv_bank bank, const uint16_t *q, int nq,
                                                               const uint16_t *wk, const uint16_t *wv, int nw,
                                                               uint16_t *out, float c, Geom g) {
  constexpr int KS = D / 16;   // K steps of S
  constexpr int DT = D / 32;   // dv tiles of O
  constexpr int RB = FCfg<D>::kRowBytes;
  const int b = blockIdx.y;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const int M = clampi(bank.budget[b], 0, g.Mcap);
  const int m = clampi(bank.occupancy[b], 0, M);
  const size_t rb = (size_t)b * g.Mcap, wb = (size_t)b * nw;
  const uint16_t *bk = static_cast<const uint16_t *>(bank.k);
  const uint16_t *bv = static_cast<const uint16_t *>(bank.v);
  __shared__ __attribute__((aligned(1024))) char kbuf[2][FCfg<D>::kTileBytes];
  __shared__ __attribute__((aligned(1024))) char vbuf[2][FCfg<D>::kTileBytes];

  const int qi = blockIdx.x * kFQ + wave * 32 + n;
  const bool qv = qi < nq;
  bf16x8 qf[KS];
  const size_t qrow = (size_t)b * nq + (qv ? qi : 0);
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4 x = {0, 0, 0, 0};
    if (qv) x = *reinterpret_cast<const u32x4 *>(q + qrow * D + 16 * kk + 8 * h);
    qf[kk] = __builtin_bit_cast(bf16x8, x);
  }
  f32x16 o[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) o[t] = f32x16{};
  float mrun = -INFINITY, lrun = 0.0f;

  // Tiles never straddle the bank/window boundary: ceil(m/64) bank tiles, then
  // ceil(nw/64) window tiles, so every tile has one (scalar) base pointer.
  const int nt0 = (m + kFK - 1) / kFK;
  const int nt = nt0 + (nw + kFK - 1) / kFK;
  auto tile_src = [&](int t, const uint16_t *&kp, const uint16_t *&vp, int &nv) {
    if (t < nt0) {
      kp = bk + (rb + (size_t)t * kFK) * D;
      vp = bv + (rb + (size_t)t * kFK) * D;
      nv = min(kFK, m - t * kFK);
    } else {
      const int tw = t - nt0;
      kp = wk + (wb + (size_t)tw * kFK) * D;
      vp = wv + (wb + (size_t)tw * kFK) * D;
      nv = min(kFK, nw - tw * kFK);
    }
  };
  const uint16_t *kp, *vp;
  int nv_cur = 0, nv_next = 0;
  if (nt > 0) {
    tile_src(0, kp, vp, nv_cur);
    ftile_issue<D>(kp, vp, nv_cur, kbuf[0], vbuf[0]);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // transposed V read: lane group gq = l / 16 (h = gq / 2), member cq = l % 16
  const int gq = l >> 4, cq = l & 15;
  for (int t = 0; t < nt; ++t) {
    const int cur = t & 1;
    if (t + 1 < nt) {
      tile_src(t + 1, kp, vp, nv_next);
      ftile_issue<D>(kp, vp, nv_next, kbuf[cur ^ 1], vbuf[cur ^ 1]);
    }
    const char *kt = kbuf[cur];
    const char *vtile = vbuf[cur];
    // S^T for two 32-key halves
    f32x16 sc[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const int key = 32 * sub + n;
      bf16x8 a[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        a[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(kt + key * RB + 16 * k_swz<D>(key, 2 * kk + h)));
      f32x16 acc = {};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk], qf[kk], acc, 0, 0, 0);
      sc[sub] = acc;
    }
    const int nvalid = nv_cur;
    if (nvalid < kFK) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (32 * sub + 8 * (i >> 2) + 4 * h + (i & 3) >= nvalid) sc[sub][i] = -INFINITY;
    }
    float tmax = sc[0][0];
#pragma unroll
    for (int i = 1; i < 16; ++i) tmax = fmaxf(tmax, sc[0][i]);
#pragma unroll
    for (int i = 0; i < 16; ++i) tmax = fmaxf(tmax, sc[1][i]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    // Lazy rescaling: the reference maximum only moves when a score exceeds it
    // by more than 2^8 in the exp2 domain, so P stays within [0, 256] and the
    // accumulated O and l are rescaled rarely (exact: the final division by l
    // removes the common factor).
    const bool grow = tmax * c > mrun * c + 8.0f;
    if (__any(grow)) {
      const float mnew = grow ? tmax : mrun;
      const float corr = __builtin_amdgcn_exp2f((mrun - mnew) * c);
      mrun = mnew;
      lrun *= corr;
#pragma unroll
      for (int t2 = 0; t2 < DT; ++t2)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[t2][i] *= corr;
    }
    const float moff = -mrun * c;
    float psum = 0.0f;
    uint32_t pb[2][8];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int i = 0; i < 16; i += 2) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[sub][i], c, moff));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[sub][i + 1], c, moff));
        psum += p0 + p1;
        pb[sub][i >> 1] = pack_bf16x2(p0, p1);
      }
    }
    lrun += psum;
    // O^T += V^T P^T
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int kst = 0; kst < 2; ++kst) {
        u32x4 bp = {pb[sub][4 * kst + 0], pb[sub][4 * kst + 1], pb[sub][4 * kst + 2], pb[sub][4 * kst + 3]};
        const bf16x8 bop = __builtin_bit_cast(bf16x8, bp);
        const int key0 = 32 * sub + 16 * kst + 4 * (gq >> 1) + (cq >> 2);
#pragma unroll
        for (int t2 = 0; t2 < DT; ++t2) {
          const int dvb = 8 * t2 + 4 * (gq & 1) + (cq & 3);  // 8-byte dv block
          const int ka = key0, kb = key0 + 8;
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4 *)(vtile + ka * RB + 16 * v_swz<D>(ka, dvb >> 1) + 8 * (dvb & 1)));
          const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4 *)(vtile + kb * RB + 16 * v_swz<D>(kb, dvb >> 1) + 8 * (dvb & 1)));
          const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
          const u32x4 av = {lo2[0], lo2[1], hi2[0], hi2[1]};
          o[t2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av), bop, o[t2], 0, 0, 0);
        }
      }
    }
    nv_cur = nv_next;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  const float ltot = lrun + __shfl_xor(lrun, 32, 64);
  if (!qv) return;
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
#pragma unroll
  for (int t2 = 0; t2 < DT; ++t2) {
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      const int dv = 32 * t2 + 8 * gg + 4 * h;
      u32x2 pk = {pack_bf16x2(o[t2][4 * gg] * inv, o[t2][4 * gg + 1] * inv),
                  pack_bf16x2(o[t2][4 * gg + 2] * inv, o[t2][4 * gg + 3] * inv)};
      *reinterpret_cast<u32x2 *>(out + qrow * D + dv) = pk;
    }
  }
}

template <int D, int DT>
hipError_t attn_impl(const dkv_bank &bank, const void *q, int nq, const void *wk, const void *wv, int nw,
                     void *out, float scale, const Geom &g, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const float scale_log2 = scale * 1.4426950408889634f;
  if constexpr (DT == DKV_BF16) {
    dim3 grid((unsigned)((nq + kFQ - 1) / kFQ), (unsigned)g.B);
    k_attn_mfma<D><<<grid, 64 * kFWaves, 0, s>>>(bank, static_cast<const uint16_t *>(q), nq,
                                                 static_cast<const uint16_t *>(wk), static_cast<const uint16_t *>(wv),
                                                 nw, static_cast<uint16_t *>(out), scale_log2, g);
  } else {
    dim3 grid((unsigned)((nq + kAThreads - 1) / kAThreads), (unsigned)g.B);
    k_attn_rowwise<D, DT><<<grid, kAThreads, 0, s>>>(bank, q, nq, wk, wv, nw, out, scale_log2, g);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const dkv_bank &bank, const void *q, int nq, const void *wk, const void *wv,
                            int nw, void *out, float scale, const Geom &g, hipStream_t s) {
  if (g.d == 128 && g.dtype == DKV_BF16) return attn_impl<128, DKV_BF16>(bank, q, nq, wk, wv, nw, out, scale, g, s);
  if (g.d == 128 && g.dtype == DKV_F32) return attn_impl<128, DKV_F32>(bank, q, nq, wk, wv, nw, out, scale, g, s);
  if (g.d == 64 && g.dtype == DKV_BF16) return attn_impl<64, DKV_BF16>(bank, q, nq, wk, wv, nw, out, scale, g, s);
  return attn_impl<64, DKV_F32>(bank, q, nq, wk, wv, nw, out, scale, g, s);
}

}  // namespace dkv
