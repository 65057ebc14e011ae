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

template <int D, int DT>
hipError_t attn_impl(const dkv_bank &bank, const void *q, int nq, const void *wk, const void *wv, int nw,
                     void *out, float scale, const Geom &g, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const float scale_log2 = scale * 1.4426950408889634f;
  dim3 grid((unsigned)((nq + kAThreads - 1) / kAThreads), (unsigned)g.B);
  k_attn_rowwise<D, DT><<<grid, kAThreads, 0, s>>>(bank, q, nq, wk, wv, nw, out, scale_log2, g);
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
