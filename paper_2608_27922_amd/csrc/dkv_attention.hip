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
//   S^T = K Q^T   A = K tile (LDS, row-major), B = Q^T (registers):
//                 lane l <-> query l % 32, registers <-> 16 keys per 32-key half,
//                 so the softmax row statistics stay inside the lane (plus one
//                 exchange with lane l ^ 32);
//   O^T += V^T P^T  B = P straight from the S registers (bf16), A = V^T read
//                 from a transposed LDS copy of the V tile.  Inside each 16-key
//                 K step the key order is permuted identically in both operands
//                 (slot 8h + j <-> key 8 (j / 4) + 4 h + j % 4), which is what
//                 the S register layout provides.
// Keys and values are staged global -> registers -> LDS with double buffering.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kFWaves = 4;
constexpr int kFQ = 32 * kFWaves;  // queries per workgroup
constexpr int kFK = 64;            // keys per tile

template <int D>
struct FCfg {
  static constexpr int kKStride = D + 8;     // bf16 per K row in LDS (odd multiple of 16 B)
  static constexpr int kVStride = kFK + 8;   // bf16 per transposed V row
  static constexpr int kKChunks = D / 8;     // 16-byte chunks per key row
  static constexpr int kKLoads = kFK * kKChunks / (64 * kFWaves);
  static constexpr int kVGroups = D / 8;     // 8-wide dv groups
  static constexpr int kVKeys = kFK * kVGroups / (64 * kFWaves);  // keys per thread (4 consecutive)
};

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16_bits(lo) | ((uint32_t)f32_to_bf16_bits(hi) << 16);
}

template <int D>
struct FStage {
  u32x4 k[FCfg<D>::kKLoads];
  u32x4 v[FCfg<D>::kVKeys];
};

template <int D>
__device__ __forceinline__ const uint16_t *key_row(const uint16_t *bk, const uint16_t *wk, size_t rb, size_t wb,
                                                   int key, int m) {
  return key < m ? bk + (rb + key) * D : wk + (wb + (key - m)) * D;
}

template <int D>
__device__ __forceinline__ void fstage_load(FStage<D> &st, const uint16_t *bk, const uint16_t *bv,
                                            const uint16_t *wk, const uint16_t *wv, size_t rb, size_t wb, int t0,
                                            int m, int total) {
#pragma unroll
  for (int q = 0; q < FCfg<D>::kKLoads; ++q) {
    const int c = threadIdx.x + q * 64 * kFWaves;
    const int key = t0 + c / FCfg<D>::kKChunks, ch = c % FCfg<D>::kKChunks;
    u32x4 x = {0, 0, 0, 0};
    if (key < total) x = *reinterpret_cast<const u32x4 *>(key_row<D>(bk, wk, rb, wb, key, m) + ch * 8);
    st.k[q] = x;
  }
  const int dg = threadIdx.x % FCfg<D>::kVGroups;
  const int kg = threadIdx.x / FCfg<D>::kVGroups;
#pragma unroll
  for (int q = 0; q < FCfg<D>::kVKeys; ++q) {
    const int key = t0 + kg * FCfg<D>::kVKeys + q;
    u32x4 x = {0, 0, 0, 0};
    if (key < total) x = *reinterpret_cast<const u32x4 *>(key_row<D>(bv, wv, rb, wb, key, m) + dg * 8);
    st.v[q] = x;
  }
}

template <int D>
__device__ __forceinline__ void fstage_store(const FStage<D> &st, uint16_t *ks, uint16_t *vt) {
#pragma unroll
  for (int q = 0; q < FCfg<D>::kKLoads; ++q) {
    const int c = threadIdx.x + q * 64 * kFWaves;
    const int key = c / FCfg<D>::kKChunks, ch = c % FCfg<D>::kKChunks;
    *reinterpret_cast<u32x4 *>(ks + key * FCfg<D>::kKStride + ch * 8) = st.k[q];
  }
  // transpose kVKeys keys x 8 dv in registers, store 8 rows of kVKeys keys
  const int dg = threadIdx.x % FCfg<D>::kVGroups;
  const int kg = threadIdx.x / FCfg<D>::kVGroups;
  constexpr int NK = FCfg<D>::kVKeys;
  static_assert(NK == 2 || NK == 4, "transposed V staging assumes 2 or 4 keys per thread");
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int w = j >> 1, sh = (j & 1) * 16;
    uint16_t *dst = vt + (dg * 8 + j) * FCfg<D>::kVStride + kg * NK;
    const uint32_t e0 = (st.v[0][w] >> sh) & 0xFFFF, e1 = (st.v[1][w] >> sh) & 0xFFFF;
    if constexpr (NK == 4) {
      const uint32_t e2 = (st.v[2][w] >> sh) & 0xFFFF, e3 = (st.v[3][w] >> sh) & 0xFFFF;
      u32x2 pk = {e0 | (e1 << 16), e2 | (e3 << 16)};
      *reinterpret_cast<u32x2 *>(dst) = pk;
    } else {
      *reinterpret_cast<uint32_t *>(dst) = e0 | (e1 << 16);
    }
  }
}

template <int D>
__global__ __launch_bounds__(64 * kFWaves, 2) void k_attn_mfma(dkv_bank bank, const uint16_t *q, int nq,
                                                               const uint16_t *wk, const uint16_t *wv, int nw,
                                                               uint16_t *out, float c, Geom g) {
  constexpr int KS = D / 16;   // K steps of S
  constexpr int DT = D / 32;   // dv tiles of O
  const int b = blockIdx.y;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const int M = clampi(bank.budget[b], 0, g.Mcap);
  const int m = clampi(bank.occupancy[b], 0, M);
  const int total = m + nw;
  const size_t rb = (size_t)b * g.Mcap, wb = (size_t)b * nw;
  const uint16_t *bk = static_cast<const uint16_t *>(bank.k);
  const uint16_t *bv = static_cast<const uint16_t *>(bank.v);
  __shared__ __attribute__((aligned(16))) uint16_t ks[2][kFK * FCfg<D>::kKStride];
  __shared__ __attribute__((aligned(16))) uint16_t vt[2][D * FCfg<D>::kVStride];

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

  const int nt = (total + kFK - 1) / kFK;
  FStage<D> st;
  if (nt > 0) {
    fstage_load<D>(st, bk, bv, wk, wv, rb, wb, 0, m, total);
    fstage_store<D>(st, ks[0], vt[0]);
  }
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    const int cur = t & 1;
    const int t0 = t * kFK;
    if (t + 1 < nt) fstage_load<D>(st, bk, bv, wk, wv, rb, wb, t0 + kFK, m, total);
    // S^T for two 32-key halves
    f32x16 sc[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const uint16_t *src = ks[cur] + (32 * sub + n) * FCfg<D>::kKStride + 8 * h;
      bf16x8 a[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) a[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(src + 16 * kk));
      f32x16 acc = {};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk], qf[kk], acc, 0, 0, 0);
      sc[sub] = acc;
    }
    const int nvalid = total - t0;
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
    const float mnew = fmaxf(mrun, tmax);
    const float corr = exp2f((mrun - mnew) * c);
    const float moff = -mnew * c;
    mrun = mnew;
    float psum = 0.0f;
    uint32_t pb[2][8];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int i = 0; i < 16; i += 2) {
        const float p0 = exp2f(__builtin_fmaf(sc[sub][i], c, moff));
        const float p1 = exp2f(__builtin_fmaf(sc[sub][i + 1], c, moff));
        psum += p0 + p1;
        pb[sub][i >> 1] = pack_bf16x2(p0, p1);
      }
    }
    lrun = lrun * corr + psum;
    if (corr != 1.0f) {
#pragma unroll
      for (int t2 = 0; t2 < DT; ++t2)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[t2][i] *= corr;
    }
    // O^T += V^T P^T
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int kst = 0; kst < 2; ++kst) {
        u32x4 bp = {pb[sub][4 * kst + 0], pb[sub][4 * kst + 1], pb[sub][4 * kst + 2], pb[sub][4 * kst + 3]};
        const bf16x8 bop = __builtin_bit_cast(bf16x8, bp);
        const int key0 = 32 * sub + 16 * kst + 4 * h;
#pragma unroll
        for (int t2 = 0; t2 < DT; ++t2) {
          const uint16_t *vr = vt[cur] + (32 * t2 + n) * FCfg<D>::kVStride + key0;
          const u32x2 lo = *reinterpret_cast<const u32x2 *>(vr);
          const u32x2 hi = *reinterpret_cast<const u32x2 *>(vr + 8);
          const u32x4 av = {lo[0], lo[1], hi[0], hi[1]};
          o[t2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av), bop, o[t2], 0, 0, 0);
        }
      }
    }
    if (t + 1 < nt) fstage_store<D>(st, ks[cur ^ 1], vt[cur ^ 1]);
    __syncthreads();
  }
  const float ltot = lrun + __shfl_xor(lrun, 32, 64);
  if (!qv) return;
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
#pragma unroll
  for (int t2 = 0; t2 < DT; ++t2) {
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int dv = 32 * t2 + 8 * gq + 4 * h;
      u32x2 pk = {pack_bf16x2(o[t2][4 * gq] * inv, o[t2][4 * gq + 1] * inv),
                  pack_bf16x2(o[t2][4 * gq + 2] * inv, o[t2][4 * gq + 3] * inv)};
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
