// DensityKV bank update and candidate scoring on gfx950.
//
// One update of every bank from one block (Supp. C, Algorithm 1) is the kernel
// sequence below, all on the caller's stream, with r* kept on the device.  The
// Gram stages of bf16 banks run on MFMA (dkv_gram_mfma.hip: k_score_mfma,
// k_gather_sorted, k_first_part_mfma, k_cross_plan, k_chunk_part_mfma,
// k_cross_mfma, k_rowsum_mfma, k_maint_mfma); fp32 banks use the
// VALU kernels of this file (k_score_gram, k_cross_gram, k_fixup, k_maint_gram).
//
//   k_begin         clamp occupancy/budget, tested prefix R of the group (Eq. 11),
//                   score scale 1/b of every bank state (Eq. 6), |k_x|^2 of
//                   every candidate, norm steps, cleared accumulators
//   score           S_x = sum_i RNE(w_ix / b_i scaled) and Wcol_x = sum_i W_ix (Eq. 6)
//   k_sort_chunks   stable ascending order of S_x, ties by source index (Alg. 1):
//   k_sort_rank     512-key chunks sorted in LDS, then ranked by search
//   crossing        prefix sums over the ordered candidates (64-candidate
//                   chunk sums), first violating prefix of every bank state (Eqs. 8-9)
//   k_feas_bank     c_r for every r and the flags c_r <= e_r (Eqs. 9-10)
//   k_feas_group    r* of each group (Eq. 11)
//   fix-up          projected density rho~(r*) of every bank state
//   k_select        mandatory + densest eviction (Sec. 3.4 step 3), commit plan
//   maintenance     weights to the evicted and to the co-admitted states (Supp. C)
//   k_commit        exact density maintenance of the survivors (Supp. C),
//                   admitted K/V placement, densities and baselines (Eq. 5)
//
// Arithmetic: keys on the 1/64 grid give exact fp32 inner products; weights are
// binary32 with round-to-nearest-even; every sum is an integer sum of Q23
// terms, so results do not depend on tiling or thread order.
#include <hip/hip_runtime.h>

#include <climits>
#include <type_traits>

#include "dkv_internal.hpp"

namespace dkv {

namespace {

constexpr int kThreads = 256;    // Gram kernels: one thread per row item
constexpr int kTile = 32;        // columns staged in LDS per step
constexpr int kBig = 1024;       // one-workgroup-per-bank kernels
constexpr uint64_t kRhoMax = (1ull << 40) - 1;

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// ---------------------------------------------------------------------------
// Block-wide scans for kBig threads (16 waves of 64 lanes).
// ---------------------------------------------------------------------------
__device__ int block_excl_scan(int v, int *total, int *tmp /*[16]*/) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) tmp[wid] = x;
  __syncthreads();
  if (wid == 0) {
    int t = lane < nw ? tmp[lane] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int y = __shfl_up(t, o, 64);
      if (lane >= o) t += y;
    }
    if (lane < nw) tmp[lane] = t;
  }
  __syncthreads();
  int pre = (wid > 0 ? tmp[wid - 1] : 0) + x - v;
  *total = tmp[nw - 1];
  __syncthreads();
  return pre;
}

__device__ int block_max(int v, int *tmp) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  if (lane == 0) tmp[wid] = v;
  __syncthreads();
  int r = tmp[0];
  for (int w = 1; w < nw; ++w) r = max(r, tmp[w]);
  __syncthreads();
  return r;
}

// Row key loaded into registers as float.
template <int D, int DT>
__device__ __forceinline__ void load_row(float (&kr)[D], const void *base, size_t row) {
#pragma unroll
  for (int j = 0; j < D; ++j) kr[j] = load_elem<DT>(base, row * D + j);
}

template <int D>
__device__ __forceinline__ float dot_row(const float (&kr)[D], const float *col) {
  float g = 0.0f;
#pragma unroll
  for (int j = 0; j < D; ++j) g = __builtin_fmaf(kr[j], col[j], g);
  return g;
}

// ---------------------------------------------------------------------------
// k_begin: grid (1 + ceil(max(N, Mcap) / 256), B).  Workgroup 0 of a bank
// clamps occupancy and budget, fixes the tested prefix R of its group (Eq. 11)
// and the score exponent E, then writes the score scale of every live state
// (Eq. 6); the other workgroups compute candidate norms, the column aug steps
// of candidates and bank states, and clear the accumulators that the Gram
// stages fill with atomic adds.
// ---------------------------------------------------------------------------
template <int D, int DT>
__global__ __launch_bounds__(kThreads) void k_begin(dkv_bank bank, const void *seg_k, const void *seg_v, Geom g,
                                                    Workspace ws, float inv_s2, int norms) {
  const int b = blockIdx.y;
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  if (blockIdx.x > 0) {
    const int j = (blockIdx.x - 1) * kThreads + threadIdx.x;
    if (j < g.N) {
      if (norms) {
        // |k|^2 (then + |v|^2 for the [K; V] geometry) in element order, 16-byte loads
        float s = 0.0f;
        if constexpr (DT == DKV_BF16) {
          for (int part = 0; part < (seg_v ? 2 : 1); ++part) {
            const uint4 *src =
                reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(part ? seg_v : seg_k) + (nb + j) * D);
            uint4 x[D / 8];
#pragma unroll
            for (int q = 0; q < D / 8; ++q) x[q] = src[q];
#pragma unroll
            for (int q = 0; q < D / 8; ++q) {
              const uint32_t w4[4] = {x[q].x, x[q].y, x[q].z, x[q].w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float lo = __uint_as_float(w4[e] << 16), hi = __uint_as_float(w4[e] & 0xFFFF0000u);
                s = __builtin_fmaf(lo, lo, s);
                s = __builtin_fmaf(hi, hi, s);
              }
            }
          }
        } else {
          const float4 *src = reinterpret_cast<const float4 *>(static_cast<const float *>(seg_k) + (nb + j) * D);
#pragma unroll 8
          for (int q = 0; q < D / 4; ++q) {
            const float4 x = src[q];
            s = __builtin_fmaf(x.x, x.x, s);
            s = __builtin_fmaf(x.y, x.y, s);
            s = __builtin_fmaf(x.z, x.z, s);
            s = __builtin_fmaf(x.w, x.w, s);
          }
        }
        ws.cnorm[nb + j] = s;
        ws.caug[nb + j] = column_aug(s, inv_s2);
      }
      ws.acol[nb + j] = 0;
      ws.sub_adm[nb + j] = 0;
      ws.mut_adm[nb + j] = 0;
    }
    if (j < g.Mcap) {
      ws.sub[rb + j] = 0;
      const int mj = clampi(bank.occupancy[b], 0, clampi(bank.budget[b], 0, g.Mcap));
      if (j < mj) ws.baug[rb + j] = column_aug(bank.knorm[rb + j], inv_s2);
    }
    return;
  }
  const int Mb = clampi(bank.budget[b], 0, g.Mcap);
  const int m = clampi(bank.occupancy[b], 0, Mb);
  // Tested prefix lengths 0..R: R = min(N, every budget of the group).
  int R = g.N;
  const int g0 = (b / g.gs) * g.gs;
  for (int j = 0; j < g.gs; ++j) R = min(R, clampi(bank.budget[g0 + j], 0, g.Mcap));
  // Score scale exponent E: binary exponent of max_i fp32(2^23 / b_i), i.e. of
  // the value at the smallest baseline (the division and rounding are monotone).
  __shared__ long long redb[kThreads / 64];
  long long mn = LLONG_MAX;
  // four independent loads per round trip
  for (int i0 = threadIdx.x; i0 < m; i0 += 4 * kThreads) {
    long long bq[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kThreads;
      const long long bv = bank.base[rb + min(i, m - 1)];  // clamped, unconditional
      bq[u] = i < m ? bv : LLONG_MAX;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) mn = bq[u] < mn ? bq[u] : mn;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const long long y = __shfl_xor(mn, o, 64);
    mn = y < mn ? y : mn;
  }
  if ((threadIdx.x & 63) == 0) redb[threadIdx.x >> 6] = mn;
  __syncthreads();
  for (int w = 0; w < kThreads / 64; ++w) mn = redb[w] < mn ? redb[w] : mn;
  int E = 0;
  if (m > 0) {
    const long long bi = mn < 1 ? 1 : mn;
    frexpf((float)(8388608.0 / (double)bi), &E);
  }
  for (int i0 = threadIdx.x; i0 < m; i0 += 4 * kThreads) {
    long long bq[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kThreads;
      bq[u] = bank.base[rb + min(i, m - 1)];  // clamped, unconditional
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kThreads;
      if (i < m) ws.bs[rb + i] = score_scale(bq[u], E);
    }
  }
  if (threadIdx.x == 0) {
    ws.m[b] = m;
    ws.M[b] = Mb;
    ws.R[b] = R;
    ws.E[b] = E;
    ws.crossed[b] = 0;
  }
}

template <int D, int DT>
void launch_begin(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p, const Workspace &ws,
                  bool norms, hipStream_t s) {
  const int span = g.N > g.Mcap ? g.N : g.Mcap;
  // [K; V] geometry: candidate norms over the concatenated key-value rows
  const void *seg_v = (p.flags & DKV_POLICY_KV_DESCRIPTOR) ? seg.v : nullptr;
  k_begin<D, DT><<<dim3((unsigned)(1 + (span + kThreads - 1) / kThreads), (unsigned)g.B), kThreads, 0, s>>>(
      bank, seg.k, seg_v, g, ws, p.inv_sigma2, norms ? 1 : 0);
}

// ---------------------------------------------------------------------------
// k_score_gram: thread = candidate x; loop over every bank state i.
// ---------------------------------------------------------------------------
template <int D, int DT>
__global__ __launch_bounds__(kThreads) void k_score_gram(dkv_bank bank, const void *seg_k, Geom g,
                                                         Prm p, Workspace ws, int64_t *out_q,
                                                         float *out_f) {
  const int b = blockIdx.y, x = blockIdx.x * kThreads + threadIdx.x;
  const int m = ws.m[b];
  const bool act = x < g.N;
  __shared__ float tk[kTile][D];
  __shared__ float tn[kTile], tb[kTile];
  float kr[D];
  float nr = 0.0f;
  if (act) {
    load_row<D, DT>(kr, seg_k, (size_t)b * g.N + x);
    nr = ws.cnorm[(size_t)b * g.N + x];
  }
  uint64_t A = 0;
  for (int i0 = 0; i0 < m; i0 += kTile) {
    const int nc = min(kTile, m - i0);
    __syncthreads();
    for (int t = threadIdx.x; t < kTile * D; t += kThreads) {
      const int c = t / D, j = t % D;
      tk[c][j] = c < nc ? load_elem<DT>(bank.k, ((size_t)b * g.Mcap + i0 + c) * D + j) : 0.0f;
    }
    if (threadIdx.x < kTile) {
      const int c = threadIdx.x;
      tn[c] = c < nc ? bank.knorm[(size_t)b * g.Mcap + i0 + c] : 0.0f;
      tb[c] = c < nc ? ws.bs[(size_t)b * g.Mcap + i0 + c] : 0.0f;
    }
    __syncthreads();
    if (act) {
      uint32_t a32 = 0;
      for (int c = 0; c < nc; ++c) {
        const float gd = dot_row<D>(kr, tk[c]);
        const float d2 = (nr + tn[c]) - 2.0f * gd;
        const float w = pair_weight(d2, p.inv_sigma2, p.p);
        a32 += q23_round(w, tb[c]);
      }
      A += a32;
    }
  }
  if (!act) return;
  const size_t o = (size_t)b * g.N + x;
  ws.acol[o] = (int64_t)A;
  if (out_q) out_q[o] = (int64_t)A;
  if (out_f) out_f[o] = m > 0 ? (float)(ldexp((double)A, ws.E[b] - 23) / (double)m) : 0.0f;
}

// ---------------------------------------------------------------------------
// Candidate order: unique keys (S_x << 13) | x sorted ascending (ties of S_x
// by source index).  k_sort_chunks: a workgroup sorts a chunk of 512 keys in
// LDS with a bitonic network (one compare-exchange per thread and stage).
// k_sort_rank: the rank of a key is its position in its own chunk plus the
// number of smaller keys in every other chunk, found by branch-free binary
// searches that run in lockstep over all chunks (ten dependent LDS rounds).
// ---------------------------------------------------------------------------
constexpr int kChunk = 512;
constexpr int kSortThreads = kChunk / 2;
constexpr int kMaxChunks = kSortMax / kChunk;

__global__ __launch_bounds__(kSortThreads) void k_sort_chunks(Geom g, Workspace ws, int64_t *out_score,
                                                              int source_order) {
  const int b = blockIdx.y, c = blockIdx.x, t = threadIdx.x;
  const size_t nb = (size_t)b * g.N;
  __shared__ uint64_t v[kChunk];
  // two keys per thread, clamped, unconditional loads
  int64_t A[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) A[u] = ws.acol[nb + min(c * kChunk + t + u * kSortThreads, g.N - 1)];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int idx = c * kChunk + t + u * kSortThreads;
    // ascending score, ties by source index; or source order alone (policy ablation)
    const uint64_t key = source_order ? (uint64_t)idx : (((uint64_t)A[u] << 13) | (uint64_t)idx);
    v[t + u * kSortThreads] = idx < g.N ? key : ~0ull;
    if (out_score && idx < g.N) out_score[nb + idx] = A[u];
  }
  __syncthreads();
  for (int k = 2; k <= kChunk; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      // the t-th index i with bit j clear, against i + j; ascending where bit k of i is clear
      const int i = ((t & ~(j - 1)) << 1) | (t & (j - 1));
      const uint64_t x = v[i], y = v[i + j];
      const bool up = (i & k) == 0;
      if (up ? (x > y) : (x < y)) {
        v[i] = y;
        v[i + j] = x;
      }
      __syncthreads();
    }
  }
  const size_t base = (size_t)b * ws.npad + (size_t)c * kChunk;
#pragma unroll
  for (int u = 0; u < 2; ++u) ws.skeys[base + t + u * kSortThreads] = v[t + u * kSortThreads];
}

template <int NCH>  // chunk slots searched (>= the number of chunks)
__global__ __launch_bounds__(kBig) void k_sort_rank(Geom g, Workspace ws, int32_t *out_order) {
  const int b = blockIdx.y;
  __shared__ uint64_t sk[kSortMax];
  const int np = ws.npad;
  const int nch = np / kChunk;
  {
    // clamped, unconditional loads, all in flight at once
    constexpr int kPer = kSortMax / kBig;
    uint64_t t[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) t[u] = ws.skeys[(size_t)b * np + min((int)threadIdx.x + u * kBig, np - 1)];
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      if ((int)threadIdx.x + u * kBig < np) sk[threadIdx.x + u * kBig] = t[u];
  }
  __syncthreads();
  const size_t nb = (size_t)b * g.N;
  for (int p = blockIdx.x * kBig + threadIdx.x; p < np; p += gridDim.x * kBig) {
    const uint64_t key = sk[p];
    if (key == ~0ull) continue;
    const int c = p / kChunk;
    // count of keys < key in every chunk: cnt grows by half while the key at
    // cnt + half - 1 is smaller (at most 511), then by one more if the key at
    // cnt is smaller; chunks past the last one read the last one and are masked
    int cnt[NCH];
#pragma unroll
    for (int c2 = 0; c2 < NCH; ++c2) cnt[c2] = 0;
#pragma unroll
    for (int half = kChunk / 2; half >= 1; half >>= 1) {
#pragma unroll
      for (int c2 = 0; c2 < NCH; ++c2) {
        const int base = min(c2, nch - 1) * kChunk;
        cnt[c2] += sk[base + cnt[c2] + half - 1] < key ? half : 0;
      }
    }
    int rank = p - c * kChunk;
#pragma unroll
    for (int c2 = 0; c2 < NCH; ++c2) {
      const int base = min(c2, nch - 1) * kChunk;
      const int n2 = cnt[c2] + (sk[base + cnt[c2]] < key ? 1 : 0);
      if (c2 < nch && c2 != c) rank += n2;
    }
    const int x = (int)(key & 0x1FFFull);
    ws.order[nb + rank] = x;
    ws.rank[nb + x] = rank;
    if (out_order) out_order[nb + rank] = x;
  }
}

// ---------------------------------------------------------------------------
// k_cross_gram: thread = bank state i; running prefix over the ordered
// candidates; first prefix length r with 2^k (rho_i + P_i(r)) >= T b_i.
// ---------------------------------------------------------------------------
template <int D, int DT>
__global__ __launch_bounds__(kThreads) void k_cross_gram(dkv_bank bank, const void *seg_k, Geom g,
                                                         Prm p, Workspace ws, int32_t *out_first) {
  const int b = blockIdx.y, i = blockIdx.x * kThreads + threadIdx.x;
  const int m = ws.m[b], R = ws.R[b];
  if ((int)blockIdx.x * kThreads >= m) return;  // uniform: no live state in this block
  const bool act = i < m;
  __shared__ float tk[kTile][D];
  __shared__ float tn[kTile];
  float kr[D];
  float nr = 0.0f;
  int64_t thr = 0;
  const size_t row = (size_t)b * g.Mcap + i;
  if (act) {
    load_row<D, DT>(kr, bank.k, row);
    nr = bank.knorm[row];
    const int64_t lim = ((int64_t)p.tau_num * bank.base[row] + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
    thr = lim - bank.rho[row];
  }
  int first = thr <= 0 ? 0 : R + 1;
  int64_t P = 0;
  uint32_t tile_sum = 0;
  for (int j0 = 0; j0 < R; j0 += kTile) {
    const int nc = min(kTile, R - j0);
    __syncthreads();
    for (int t = threadIdx.x; t < kTile * D; t += kThreads) {
      const int c = t / D, j = t % D;
      float v = 0.0f;
      if (c < nc) {
        const int x = ws.order[(size_t)b * g.N + j0 + c];
        v = load_elem<DT>(seg_k, ((size_t)b * g.N + x) * D + j);
      }
      tk[c][j] = v;
    }
    if (threadIdx.x < kTile) {
      const int c = threadIdx.x;
      tn[c] = c < nc ? ws.cnorm[(size_t)b * g.N + ws.order[(size_t)b * g.N + j0 + c]] : 0.0f;
    }
    __syncthreads();
    if (act) {
      for (int c = 0; c < nc; ++c) {
        const float gd = dot_row<D>(kr, tk[c]);
        const float d2 = (nr + tn[c]) - 2.0f * gd;
        const uint32_t W = q23_round(pair_weight(d2, p.inv_sigma2, p.p), 8388608.0f);
        P += W;
        tile_sum += W;
        if (first > R && P >= thr) first = j0 + c + 1;
        const int done = j0 + c + 1;
        if ((done % kCkStride) == 0) {
          ws.ck[row * ws.nck + (done / kCkStride - 1)] = tile_sum;
          tile_sum = 0;
        }
      }
    }
  }
  if (!act) return;
  ws.first[row] = first;
  if (out_first) out_first[row] = first;
}

// ---------------------------------------------------------------------------
// k_feasible: one workgroup per group.  c_r = #{i : first_i <= r}; feasible
// iff c_r <= e_r for every bank of the group; r* = largest feasible r.
// ---------------------------------------------------------------------------
__device__ void block_inclusive_scan_lds(int *a, int n, int *tmp) {
  const int per = (n + kBig - 1) / kBig;
  const int lo = min(n, (int)threadIdx.x * per), hi = min(n, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += a[i];
  int tot;
  int pre = block_excl_scan(s, &tot, tmp);
  for (int i = lo; i < hi; ++i) {
    pre += a[i];
    a[i] = pre;
  }
  __syncthreads();
}

// Per bank: c_r = #{i : first_i <= r} by histogram + scan, and bit r of the
// feasibility mask set iff c_r <= e_r = max(0, m + r - M) (Eqs. 9-10).
__global__ __launch_bounds__(kBig) void k_feas_bank(Geom g, Workspace ws) {
  const int b = blockIdx.x;
  __shared__ int hist[kSortMax + 1];
  __shared__ int tmp[16];
  const int R = ws.R[b];
  const int m = ws.m[b], M = ws.M[b];
  for (int r = threadIdx.x; r <= R; r += kBig) hist[r] = 0;
  __syncthreads();
  // four independent (clamped, unconditional) loads per round trip
  for (int i0 = threadIdx.x; i0 < m; i0 += 4 * kBig) {
    int t[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) t[u] = ws.first[(size_t)b * g.Mcap + min(i0 + u * kBig, m - 1)];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i0 + u * kBig < m && t[u] <= R) atomicAdd(&hist[t[u]], 1);
  }
  __syncthreads();
  block_inclusive_scan_lds(hist, R + 1, tmp);
  // one wave per 64 values of r: the flags by ballot, two mask words per wave
  uint32_t *f = ws.feas + (size_t)b * ws.nfw;
  const int lane = threadIdx.x & 63;
  for (int w2 = threadIdx.x >> 6; 2 * w2 < ws.nfw; w2 += kBig / 64) {
    const int r = 64 * w2 + lane;
    const bool ok = r <= R && hist[r <= R ? r : 0] <= max(0, m + r - M);
    const unsigned long long bits = __ballot(ok);
    if (lane == 0) f[2 * w2] = (uint32_t)bits;
    if (lane == 1 && 2 * w2 + 1 < ws.nfw) f[2 * w2 + 1] = (uint32_t)(bits >> 32);
  }
}

// Per group: r* = the largest r feasible for every bank of the group (Eq. 11).
__global__ __launch_bounds__(kBig) void k_feas_group(Geom g, Workspace ws, int32_t *out_rstar) {
  constexpr int kMaxWords = (DKV_MAX_CANDIDATES + 1 + 31) / 32;
  const int grp = blockIdx.x;
  __shared__ int tmp[16];
  __shared__ uint32_t mask[kMaxWords];
  const int b0 = grp * g.gs;
  const int nfw = ws.nfw, tot = g.gs * nfw;
  for (int w = threadIdx.x; w < nfw; w += kBig) mask[w] = ~0u;
  __syncthreads();
  // the group's masks are consecutive (bank j of the group, word w at j * nfw + w):
  // AND them into LDS, four independent (clamped, unconditional) loads per round trip
  const uint32_t *gf = ws.feas + (size_t)b0 * nfw;
  for (int i0 = threadIdx.x; i0 < tot; i0 += 4 * kBig) {
    uint32_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = gf[min(i0 + u * kBig, tot - 1)];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i0 + u * kBig < tot) atomicAnd(&mask[(i0 + u * kBig) % nfw], v[u]);
  }
  __syncthreads();
  int best = 0;
  for (int w = threadIdx.x; w < nfw; w += kBig) {
    const uint32_t bits = mask[w];
    if (bits) best = max(best, 32 * w + 31 - __clz(bits));
  }
  best = block_max(best, tmp);
  if (threadIdx.x == 0) {
    ws.r_star[grp] = best;
    if (out_rstar) out_rstar[grp] = best;
  }
  for (int j = threadIdx.x; j < g.gs; j += kBig) {
    const int b = b0 + j;
    ws.e[b] = max(0, ws.m[b] + best - ws.M[b]);
  }
}

// ---------------------------------------------------------------------------
// k_fixup: rho~_i(r*) = rho_i + the whole 64-candidate chunk sums before r*
// + the partial chunk.
// ---------------------------------------------------------------------------
template <int D, int DT>
__global__ __launch_bounds__(kThreads) void k_fixup(dkv_bank bank, const void *seg_k, Geom g, Prm p,
                                                    Workspace ws, int64_t *out_rho_t) {
  const int b = blockIdx.y, i = blockIdx.x * kThreads + threadIdx.x;
  const int m = ws.m[b];
  if ((int)blockIdx.x * kThreads >= m) return;
  const bool act = i < m;
  const int rs = ws.r_star[b / g.gs];
  const int full = rs / kCkStride;
  __shared__ float tk[kTile][D];
  __shared__ float tn[kTile];
  float kr[D];
  float nr = 0.0f;
  int64_t P = 0;
  const size_t row = (size_t)b * g.Mcap + i;
  if (act) {
    load_row<D, DT>(kr, bank.k, row);
    nr = bank.knorm[row];
    for (int t = 0; t < full; ++t) P += ws.ck[row * ws.nck + t];
  }
  for (int j0 = full * kCkStride; j0 < rs; j0 += kTile) {
    const int nc = min(kTile, rs - j0);
    __syncthreads();
    for (int t = threadIdx.x; t < kTile * D; t += kThreads) {
      const int c = t / D, j = t % D;
      float v = 0.0f;
      if (c < nc) {
        const int x = ws.order[(size_t)b * g.N + j0 + c];
        v = load_elem<DT>(seg_k, ((size_t)b * g.N + x) * D + j);
      }
      tk[c][j] = v;
    }
    if (threadIdx.x < kTile) {
      const int c = threadIdx.x;
      tn[c] = c < nc ? ws.cnorm[(size_t)b * g.N + ws.order[(size_t)b * g.N + j0 + c]] : 0.0f;
    }
    __syncthreads();
    if (act) {
      for (int c = 0; c < nc; ++c) {
        const float gd = dot_row<D>(kr, tk[c]);
        const float d2 = (nr + tn[c]) - 2.0f * gd;
        P += q23_round(pair_weight(d2, p.inv_sigma2, p.p), 8388608.0f);
      }
    }
  }
  if (!act) return;
  const int64_t rt = bank.rho[row] + P;
  ws.rho_t[row] = rt;
  if (out_rho_t) out_rho_t[row] = rt;
}

// ---------------------------------------------------------------------------
// k_select: one workgroup per bank.  Violators at r* are evicted; the fill
// takes the non-violators with the largest rho~(r*), ties by provenance, then
// slot (key (2^40-1-rho~, prov, slot) ascending, found by MSB radix select).
// Then the commit plan: evicted list, admitted list, final slot of everything.
// ---------------------------------------------------------------------------
enum : unsigned char { ST_NONE = 0, ST_CAND = 1, ST_SEL = 2, ST_VIOL = 3 };

__device__ __forceinline__ int sel_digit(const Workspace &ws, const dkv_bank &bank, size_t row, int slot,
                                         int pass) {
  if (pass < 5) {
    const uint64_t w0 = kRhoMax - (uint64_t)ws.rho_t[row];
    return (int)((w0 >> (8 * (4 - pass))) & 0xFF);
  }
  if (pass < 13) {
    const uint64_t w1 = (uint64_t)bank.prov[row];
    return (int)((w1 >> (8 * (12 - pass))) & 0xFF);
  }
  return (int)(((uint32_t)slot >> (8 * (14 - pass))) & 0xFF);
}

__global__ __launch_bounds__(kBig) void k_select(dkv_bank bank, Geom g, Workspace ws,
                                                 dkv_update_out out, uint32_t flags) {
  // policy ablations: no mandatory set, or a fill in admission order (key
  // (provenance, slot): the radix passes over rho~ are skipped)
  const bool no_mandatory = (flags & DKV_POLICY_DENSEST_ONLY) != 0;
  const int first_pass = (flags & DKV_POLICY_SOURCE_FILL) ? 5 : 0;
  const int b = blockIdx.x;
  const int m = ws.m[b];
  const int rs = ws.r_star[b / g.gs];
  const int e = ws.e[b];
  __shared__ unsigned char st[DKV_MAX_CAPACITY + 1];
  __shared__ int hist[256];
  __shared__ int tmp[16];
  __shared__ int sh_bucket, sh_below, sh_cnt;
  const size_t rb = (size_t)b * g.Mcap;

  // this thread's candidate ranks (admitted list below), loaded up front
  const int N = g.N;
  const size_t nb = (size_t)b * N;
  constexpr int kPerN = (DKV_MAX_CANDIDATES + kBig - 1) / kBig;
  const int perN = (N + kBig - 1) / kBig;
  const int loN = min(N, (int)threadIdx.x * perN), hiN = min(N, loN + perN);
  int rk[kPerN];
#pragma unroll
  for (int u = 0; u < kPerN; ++u) {
    const int r = N > 0 ? ws.rank[nb + min(loN + u, N - 1)] : INT_MAX;  // clamped, unconditional
    rk[u] = loN + u < hiN ? r : INT_MAX;
  }
  // violators and candidates for the fill (four independent loads per round trip)
  int nv_local = 0;
  for (int i0 = threadIdx.x; i0 < m; i0 += 4 * kBig) {
    int f[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) f[u] = ws.first[rb + min(i0 + u * kBig, m - 1)];  // clamped, unconditional
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kBig;
      if (i < m) {
        const bool v = !no_mandatory && f[u] <= rs;
        st[i] = v ? ST_VIOL : ST_CAND;
        nv_local += v;
      }
    }
  }
  int nv;
  (void)block_excl_scan(nv_local, &nv, tmp);
  int need = e - nv;
  if (need > 0 && need >= m - nv) {
    // every non-violator is evicted too (e = m): no ranking needed
    for (int i = threadIdx.x; i < m; i += kBig)
      if (st[i] == ST_CAND) st[i] = ST_SEL;
    need = 0;
    __syncthreads();
  }
  if (need > 0) {
    for (int pass = first_pass; pass < 15; ++pass) {
      for (int t = threadIdx.x; t < 256; t += kBig) hist[t] = 0;
      __syncthreads();
      for (int i = threadIdx.x; i < m; i += kBig)
        if (st[i] == ST_CAND) atomicAdd(&hist[sel_digit(ws, bank, rb + i, i, pass)], 1);
      __syncthreads();
      if (threadIdx.x == 0) {
        int cum = 0, d = 0;
        while (d < 255 && cum + hist[d] < need) cum += hist[d++];
        sh_bucket = d;
        sh_below = cum;
        sh_cnt = hist[d];
      }
      __syncthreads();
      const int bk = sh_bucket, below = sh_below, cnt = sh_cnt;
      const bool finish = (need - below) == cnt;
      for (int i = threadIdx.x; i < m; i += kBig) {
        if (st[i] != ST_CAND) continue;
        const int dg = sel_digit(ws, bank, rb + i, i, pass);
        if (dg < bk || (dg == bk && finish)) st[i] = ST_SEL;
        else if (dg > bk) st[i] = ST_NONE;
      }
      need -= below;
      __syncthreads();
      if (finish) break;
    }
  }

  // evicted list (ascending slots) and rank of each evicted slot
  const int per = (m + kBig - 1) / kBig;
  const int lo = min(m, (int)threadIdx.x * per), hi = min(m, lo + per);
  int cnt_local = 0;
  for (int i = lo; i < hi; ++i) cnt_local += (st[i] == ST_VIOL || st[i] == ST_SEL);
  int n_ev;
  int pos = block_excl_scan(cnt_local, &n_ev, tmp);
  int spos = lo - pos;  // survivors before this thread's range
  for (int i = lo; i < hi; ++i) {
    if (st[i] == ST_VIOL || st[i] == ST_SEL) {
      ws.ev_list[rb + pos] = i;
      ws.dest[rb + i] = -1 - pos;  // provisional: encodes the evicted rank
      if (pos < rs) ws.adm_dest[nb + pos] = i;  // admitted entry pos fills the pos-th evicted slot
      ++pos;
    } else {
      ws.surv_list[rb + spos] = i;
      ws.dest[rb + i] = i;
      ++spos;
    }
  }
  // admitted list: source indices x with rank(x) < r*, ascending; entries
  // beyond the evicted slots are appended after the old occupancy
  int ca = 0;
#pragma unroll
  for (int u = 0; u < kPerN; ++u) ca += rk[u] < rs;
  int n_adm;
  int pa = block_excl_scan(ca, &n_adm, tmp);
  __syncthreads();
  const int m_new = m - n_ev + rs;
#pragma unroll
  for (int u = 0; u < kPerN; ++u) {
    if (rk[u] < rs) {
      ws.adm_list[nb + pa] = loN + u;
      if (pa >= n_ev) ws.adm_dest[nb + pa] = m + (pa - n_ev);
      ++pa;
    }
  }
  __syncthreads();
  if (n_ev > rs) {
    // More evicted than admitted: close the holes below m_new with the
    // occupants at or beyond m_new, both in ascending slot order.
    // occupied(s) after placement: survivor, or an evicted slot filled by an
    // admitted candidate (evicted rank < r*).
    int mv_local = 0, lh_local = 0;
    for (int i = lo; i < hi; ++i) {
      const int dsl = ws.dest[rb + i];
      const bool occ = dsl >= 0 || (-1 - dsl) < rs;
      mv_local += occ && i >= m_new;
      lh_local += !occ && i < m_new;
    }
    int n_mv, n_lh;
    int pm = block_excl_scan(mv_local, &n_mv, tmp);
    int ph = block_excl_scan(lh_local, &n_lh, tmp);
    // list of the holes below m_new, ascending
    for (int i = lo; i < hi; ++i) {
      const int dsl = ws.dest[rb + i];
      const bool occ = dsl >= 0 || (-1 - dsl) < rs;
      if (!occ && i < m_new) ws.hole_list[rb + (ph++)] = i;
    }
    __syncthreads();
    for (int i = lo; i < hi; ++i) {
      const int dsl = ws.dest[rb + i];
      const bool occ = dsl >= 0 || (-1 - dsl) < rs;
      if (occ && i >= m_new) {
        const int to = ws.hole_list[rb + pm];
        ++pm;
        if (dsl >= 0) {
          ws.dest[rb + i] = to;  // moving survivor
        } else {
          ws.adm_dest[nb + (-1 - dsl)] = to;  // admitted candidate placed in a high hole
        }
      }
    }
    __syncthreads();
  }
  // finalize dest: evicted -> -1; outputs
  for (int i = lo; i < hi; ++i)
    if (ws.dest[rb + i] < 0) ws.dest[rb + i] = -1;
  if (out.evicted) {
    for (int j = threadIdx.x; j < g.Mcap; j += kBig) out.evicted[rb + j] = j < n_ev ? ws.ev_list[rb + j] : -1;
  }
  if (out.admitted) {
    for (int j = threadIdx.x; j < N; j += kBig) out.admitted[nb + j] = j < n_adm ? ws.adm_list[nb + j] : -1;
  }
  if (threadIdx.x == 0) {
    ws.n_ev[b] = n_ev;
    ws.m_new[b] = m_new;
    bank.occupancy[b] = m_new;
    if (out.n_evicted) out.n_evicted[b] = n_ev;
    if (out.n_admitted) out.n_admitted[b] = rs;
  }
}

// ---------------------------------------------------------------------------
// k_maint_gram: virtual rows [0, Mcap) = pre-update slots (survivors),
// [Mcap, Mcap + N) = admitted list entries.  Survivors: sum of weights to the
// evicted states.  Admitted: sum of weights to the survivors and to the other
// admitted candidates (self excluded by index).
// ---------------------------------------------------------------------------
template <int D, int DT>
__global__ __launch_bounds__(kThreads) void k_maint_gram(dkv_bank bank, const void *seg_k, Geom g,
                                                         Prm p, Workspace ws) {
  const int b = blockIdx.y, v = blockIdx.x * kThreads + threadIdx.x;
  const int m = ws.m[b], n_ev = ws.n_ev[b];
  const int n_surv = m - n_ev;
  const int rs = ws.r_star[b / g.gs];
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  bool surv = false, adm = false;
  if (v < g.Mcap) surv = v < m && ws.dest[rb + v] >= 0;
  else adm = (v - g.Mcap) < rs && (v - g.Mcap) < g.N;
  const bool act = surv || adm;
  if (!__syncthreads_or(act)) return;
  const bool any_adm = __syncthreads_or(adm);
  const bool any_surv = __syncthreads_or(surv);
  __shared__ float tk[kTile][D];
  __shared__ float tn[kTile];
  float kr[D];
  float nr = 0.0f;
  const int k_adm = v - g.Mcap;
  if (surv) {
    load_row<D, DT>(kr, bank.k, rb + v);
    nr = bank.knorm[rb + v];
  } else if (adm) {
    const int x = ws.adm_list[nb + k_adm];
    load_row<D, DT>(kr, seg_k, nb + x);
    nr = ws.cnorm[nb + x];
  }
  // pass 0: evicted columns (survivor rows)
  // pass 1: survivor columns (admitted rows)
  // pass 2: admitted columns (admitted rows)
  int64_t s_base = 0, s_adm = 0;
  for (int pass = 0; pass < 3; ++pass) {
    int ncol;
    if (pass == 0) ncol = any_surv ? n_ev : 0;
    else if (pass == 1) ncol = any_adm ? n_surv : 0;
    else ncol = any_adm ? rs : 0;
    const bool use = pass == 0 ? surv : adm;
    for (int j0 = 0; j0 < ncol; j0 += kTile) {
      const int nc = min(kTile, ncol - j0);
      __syncthreads();
      for (int t = threadIdx.x; t < kTile * D; t += kThreads) {
        const int c = t / D, j = t % D;
        float val = 0.0f;
        if (c < nc) {
          if (pass == 0) val = load_elem<DT>(bank.k, (rb + ws.ev_list[rb + j0 + c]) * D + j);
          else if (pass == 1) val = load_elem<DT>(bank.k, (rb + ws.surv_list[rb + j0 + c]) * D + j);
          else val = load_elem<DT>(seg_k, (nb + ws.adm_list[nb + j0 + c]) * D + j);
        }
        tk[c][j] = val;
      }
      if (threadIdx.x < kTile) {
        const int c = threadIdx.x;
        float nv = 0.0f;
        if (c < nc) {
          if (pass == 0) nv = bank.knorm[rb + ws.ev_list[rb + j0 + c]];
          else if (pass == 1) nv = bank.knorm[rb + ws.surv_list[rb + j0 + c]];
          else nv = ws.cnorm[nb + ws.adm_list[nb + j0 + c]];
        }
        tn[c] = nv;
      }
      __syncthreads();
      if (use) {
        for (int c = 0; c < nc; ++c) {
          if (pass == 2 && j0 + c == k_adm) continue;  // j != x by index
          const float d2 = (nr + tn[c]) - 2.0f * dot_row<D>(kr, tk[c]);
          const uint32_t W = q23_round(pair_weight(d2, p.inv_sigma2, p.p), 8388608.0f);
          if (pass == 2) s_adm += W;
          else s_base += W;
        }
      }
    }
  }
  if (surv) ws.sub[rb + v] = s_base;
  if (adm) {
    ws.sub_adm[nb + k_adm] = s_base;
    ws.mut_adm[nb + k_adm] = s_adm;
  }
}

// ---------------------------------------------------------------------------
// Commit.  commit_surv: thread per surviving state: rho <- rho~(r*) minus its
// weights to the evicted states (Supp. C); a state that closes a hole (only when
// more states left than entered) moves with its key, value and metadata.
// commit_adm: the admitted K/V rows into their slots, four 16-byte chunks of
// one token per thread; the first lane of each token writes its density over
// the final bank, frozen baseline max(rho, delta) (Eq. 5), provenance and norm.
// ---------------------------------------------------------------------------
template <int D, int DT>
__device__ __forceinline__ void commit_surv(const dkv_bank &bank, const Geom &g, const Prm &p, const Workspace &ws,
                                            int bx) {
  using E = typename std::conditional<DT == DKV_BF16, uint16_t, float>::type;
  const int b = blockIdx.y, v = bx * kThreads + threadIdx.x;
  if (v >= ws.m[b]) return;
  const size_t rb = (size_t)b * g.Mcap;
  const int to = ws.dest[rb + v];
  if (to < 0) return;
  const int64_t rho = ws.rho_t[rb + v] - ws.sub[rb + v];
  if (to != v) {
    E *K = static_cast<E *>(bank.k);
    E *V = static_cast<E *>(bank.v);
    for (int j = 0; j < D; ++j) {
      K[(rb + to) * D + j] = K[(rb + v) * D + j];
      V[(rb + to) * D + j] = V[(rb + v) * D + j];
    }
    bank.base[rb + to] = bank.base[rb + v];
    bank.prov[rb + to] = bank.prov[rb + v];
    bank.knorm[rb + to] = bank.knorm[rb + v];
  }
  bank.rho[rb + to] = rho;
  // refreshed baselines (policy ablation): b = max(rho, delta) after the update
  if (p.flags & DKV_POLICY_REFRESH_BASE) bank.base[rb + to] = rho > p.delta_q ? rho : p.delta_q;
}

typedef uint32_t vu4 __attribute__((ext_vector_type(4)));
constexpr int kCommitChunks = 4;  // 16-byte chunks of one admitted token per thread (1 and 2 were slower)

// Admitted tokens per workgroup of the commit: a token's K and V rows are
// 2 * D * sizeof(E) / 16 chunks, kCommitChunks per thread.
template <int D, int DT>
__host__ __device__ constexpr int commit_tok_per_wg() {
  return kThreads / (2 * D * (DT == DKV_BF16 ? 2 : 4) / 16 / kCommitChunks);
}

template <int D, int DT>
__device__ __forceinline__ void commit_adm(const dkv_bank &bank, const dkv_segment &seg, const Geom &g,
                                           const Prm &p, const Workspace &ws, int bx) {
  using E = typename std::conditional<DT == DKV_BF16, uint16_t, float>::type;
  constexpr int kCh = D * (int)sizeof(E) / 16;  // 16-byte chunks per key (and per value) row
  constexpr int kLanes = 2 * kCh / kCommitChunks;  // lanes per token
  constexpr int kTokWG = commit_tok_per_wg<D, DT>();
  static_assert(2 * kCh % kCommitChunks == 0 && kThreads % kLanes == 0, "whole tokens per workgroup");
  const int b = blockIdx.y;
  const int j = threadIdx.x % kLanes;
  const int k = bx * kTokWG + threadIdx.x / kLanes;
  const int rs = min(ws.r_star[b / g.gs], g.N);
  const size_t rb = (size_t)b * g.Mcap, nb = (size_t)b * g.N;
  if (bx * kTokWG >= rs) return;  // whole workgroup
  // loads from a clamped (in-range) entry, unconditional so that they overlap;
  // only the stores are predicated
  const int kc = min(k, rs - 1);
  const int x = ws.adm_list[nb + kc], to = ws.adm_dest[nb + kc];
  vu4 tmp[kCommitChunks];
#pragma unroll
  for (int u = 0; u < kCommitChunks; ++u) {
    const int cc = j + kLanes * u;  // chunk of the token's [K row; V row]
    const bool isv = cc >= kCh;
    tmp[u] = reinterpret_cast<const vu4 *>(static_cast<const E *>(isv ? seg.v : seg.k) + (nb + x) * D)[cc - (isv ? kCh : 0)];
  }
  if (k >= rs) return;
#pragma unroll
  for (int u = 0; u < kCommitChunks; ++u) {
    const int cc = j + kLanes * u;
    const bool isv = cc >= kCh;
    // streaming store: the bank rows are not read again by this update
    __builtin_nontemporal_store(tmp[u], reinterpret_cast<vu4 *>(static_cast<E *>(isv ? bank.v : bank.k) + (rb + to) * D) +
                                            (cc - (isv ? kCh : 0)));
  }
  if (j == 0) {
    // density over the final bank: the survivors plus the other co-admitted candidates
    const int64_t rho = ws.sub_adm[nb + k] + ws.mut_adm[nb + k];
    bank.rho[rb + to] = rho;
    bank.base[rb + to] = rho > p.delta_q ? rho : p.delta_q;
    bank.prov[rb + to] = ((int64_t)p.block_id << 32) | (int64_t)x;
    bank.knorm[rb + to] = ws.cnorm[nb + x];
  }
}

// Commit (Eq. 12) in one launch: the first nx_surv workgroups update the
// survivors (and move the few that close holes), the rest place the admitted
// candidates.  The two write disjoint slots.
template <int D, int DT>
__global__ __launch_bounds__(kThreads) void k_commit(dkv_bank bank, dkv_segment seg, Geom g, Prm p, Workspace ws,
                                                     int nx_surv) {
  if ((int)blockIdx.x < nx_surv) commit_surv<D, DT>(bank, g, p, ws, blockIdx.x);
  else commit_adm<D, DT>(bank, seg, g, p, ws, blockIdx.x - nx_surv);
}

// ---------------------------------------------------------------------------
// k_bank_density: Phi over the bank of every live slot, from scratch (Eq. 3).
// ---------------------------------------------------------------------------
template <int D, int DT>
__global__ __launch_bounds__(kThreads) void k_bank_density(dkv_bank bank, Geom g, Prm p, Workspace ws,
                                                           int64_t *out) {
  const int b = blockIdx.y, i = blockIdx.x * kThreads + threadIdx.x;
  const int m = ws.m[b];
  if ((int)blockIdx.x * kThreads >= m) return;
  const bool act = i < m;
  const size_t rb = (size_t)b * g.Mcap;
  __shared__ float tk[kTile][D];
  __shared__ float tn[kTile];
  float kr[D];
  float nr = 0.0f;
  if (act) {
    load_row<D, DT>(kr, bank.k, rb + i);
    nr = bank.knorm[rb + i];
  }
  int64_t s = 0;
  for (int j0 = 0; j0 < m; j0 += kTile) {
    const int nc = min(kTile, m - j0);
    __syncthreads();
    for (int t = threadIdx.x; t < kTile * D; t += kThreads) {
      const int c = t / D, j = t % D;
      tk[c][j] = c < nc ? load_elem<DT>(bank.k, (rb + j0 + c) * D + j) : 0.0f;
    }
    if (threadIdx.x < kTile) tn[threadIdx.x] = (int)threadIdx.x < nc ? bank.knorm[rb + j0 + threadIdx.x] : 0.0f;
    __syncthreads();
    if (act) {
      for (int c = 0; c < nc; ++c) {
        if (j0 + c == i) continue;  // j != i by index
        const float d2 = (nr + tn[c]) - 2.0f * dot_row<D>(kr, tk[c]);
        s += q23_round(pair_weight(d2, p.inv_sigma2, p.p), 8388608.0f);
      }
    }
  }
  if (act) out[rb + i] = s;
}

__global__ void k_pair_weight(const float *d2, int64_t n, Prm p, int32_t *w) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) w[i] = (int32_t)q23_round(pair_weight(d2[i], p.inv_sigma2, p.p), 8388608.0f);
}

inline dim3 grid2(int n, int per, int B) { return dim3((unsigned)((n + per - 1) / per), (unsigned)B); }

template <int D, int DT>
hipError_t update_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                       const dkv_update_out *outp, const Workspace &ws, hipStream_t s) {
  dkv_update_out out = outp ? *outp : dkv_update_out{};
  // bf16 banks: Gram stages on MFMA; fp32 banks: the same stages on the VALU.
  constexpr bool kMfma = DT == DKV_BF16;
  launch_begin<D, DT>(bank, seg, g, p, ws, g.N > 0, s);
  if (g.N > 0) {
    if (kMfma) launch_gram_mfma(bank, seg, g, p, out, ws, s, 0);
    else k_score_gram<D, DT><<<grid2(g.N, kThreads, g.B), kThreads, 0, s>>>(bank, seg.k, g, p, ws, nullptr, nullptr);
    k_sort_chunks<<<dim3((unsigned)((g.N + kChunk - 1) / kChunk), (unsigned)g.B), kSortThreads, 0, s>>>(
        g, ws, out.score_q, (p.flags & DKV_POLICY_SOURCE_ORDER) ? 1 : 0);
    {
      const dim3 grid((unsigned)((ws.npad + kBig - 1) / kBig), (unsigned)g.B);
      const int nch = ws.npad / kChunk;
      if (nch <= 4) k_sort_rank<4><<<grid, kBig, 0, s>>>(g, ws, out.order);
      else if (nch <= 8) k_sort_rank<8><<<grid, kBig, 0, s>>>(g, ws, out.order);
      else if (nch <= 12) k_sort_rank<12><<<grid, kBig, 0, s>>>(g, ws, out.order);
      else k_sort_rank<kMaxChunks><<<grid, kBig, 0, s>>>(g, ws, out.order);
    }
  }
  // within-block sequential competition: the rest is one candidate per step
  if (kMfma && (p.flags & DKV_POLICY_SEQUENTIAL)) return launch_sequential(bank, seg, g, p, out, ws, s);
  if (g.N > 0 && kMfma) launch_gram_mfma(bank, seg, g, p, out, ws, s, 4);
  // with no candidates only states that already violate are found (prefix 0)
  if (kMfma) launch_gram_mfma(bank, seg, g, p, out, ws, s, 1);
  else k_cross_gram<D, DT><<<grid2(g.Mcap, kThreads, g.B), kThreads, 0, s>>>(bank, seg.k, g, p, ws, out.first_cross);
  k_feas_bank<<<g.B, kBig, 0, s>>>(g, ws);
  k_feas_group<<<g.G, kBig, 0, s>>>(g, ws, out.r_star);
  if (kMfma) launch_gram_mfma(bank, seg, g, p, out, ws, s, 2);
  else k_fixup<D, DT><<<grid2(g.Mcap, kThreads, g.B), kThreads, 0, s>>>(bank, seg.k, g, p, ws, out.rho_tilde);
  k_select<<<g.B, kBig, 0, s>>>(bank, g, ws, out, p.flags);
  if (kMfma) launch_gram_mfma(bank, seg, g, p, out, ws, s, 3);
  else k_maint_gram<D, DT><<<grid2(g.Mcap + g.N, kThreads, g.B), kThreads, 0, s>>>(bank, seg.k, g, p, ws);
  {
    const int nxs = (g.Mcap + kThreads - 1) / kThreads;
    const int tok_per_wg = commit_tok_per_wg<D, DT>();
    const int nxa = g.N > 0 ? (g.N + tok_per_wg - 1) / tok_per_wg : 0;
    k_commit<D, DT><<<dim3((unsigned)(nxs + nxa), (unsigned)g.B), kThreads, 0, s>>>(bank, seg, g, p, ws, nxs);
  }
  return hipGetLastError();
}

template <int D, int DT>
hipError_t score_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                      int64_t *score_q, float *score_f, int64_t *density, const Workspace &ws,
                      hipStream_t s) {
  launch_begin<D, DT>(bank, seg, g, p, ws, g.N > 0 && (score_q || score_f), s);
  if constexpr (DT == DKV_BF16) {
    launch_score_mfma(bank, seg, g, p, (g.N > 0) ? score_q : nullptr, (g.N > 0) ? score_f : nullptr, density, ws, s);
  } else {
    if (g.N > 0 && (score_q || score_f))
      k_score_gram<D, DT><<<grid2(g.N, kThreads, g.B), kThreads, 0, s>>>(bank, seg.k, g, p, ws, score_q, score_f);
    if (density)
      k_bank_density<D, DT><<<grid2(g.Mcap, kThreads, g.B), kThreads, 0, s>>>(bank, g, p, ws, density);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_update(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                         const dkv_update_out *out, const Workspace &ws, hipStream_t s) {
  if (g.d == 128 && g.dtype == DKV_BF16) return update_impl<128, DKV_BF16>(bank, seg, g, p, out, ws, s);
  if (g.d == 128 && g.dtype == DKV_F32) return update_impl<128, DKV_F32>(bank, seg, g, p, out, ws, s);
  if (g.d == 64 && g.dtype == DKV_BF16) return update_impl<64, DKV_BF16>(bank, seg, g, p, out, ws, s);
  return update_impl<64, DKV_F32>(bank, seg, g, p, out, ws, s);
}

hipError_t launch_score(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                        int64_t *score_q, float *score_f, int64_t *density, const Workspace &ws,
                        hipStream_t s) {
  if (g.d == 128 && g.dtype == DKV_BF16) return score_impl<128, DKV_BF16>(bank, seg, g, p, score_q, score_f, density, ws, s);
  if (g.d == 128 && g.dtype == DKV_F32) return score_impl<128, DKV_F32>(bank, seg, g, p, score_q, score_f, density, ws, s);
  if (g.d == 64 && g.dtype == DKV_BF16) return score_impl<64, DKV_BF16>(bank, seg, g, p, score_q, score_f, density, ws, s);
  return score_impl<64, DKV_F32>(bank, seg, g, p, score_q, score_f, density, ws, s);
}

hipError_t launch_pair_weight(const float *d2, int64_t n, const Prm &p, int32_t *w, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  k_pair_weight<<<(unsigned)blocks, 256, 0, s>>>(d2, n, p, w);
  return hipGetLastError();
}

}  // namespace dkv
