// Within-block sequential competition (Supp. E, "Within-block competition";
// DKV_POLICY_SEQUENTIAL in include/densitykv.h): the candidates of a block are
// offered one at a time, in the order fixed at the start of the block, and
// every step is decided against the banks as the earlier steps left them.
//
//   k_seq_gram    W between every pair of items of a bank, the items being its
//                 slots 0..Mcap-1 (pre-update states) and its candidates, on
//                 bf16 MFMA (32 x 32 tiles, one per wave), stored as
//                 [B, L, L] uint32 with L = Mcap + N
//   k_seq         one workgroup per group, one wave per bank (a wave takes
//                 every bank_index % waves): for every step the one-candidate
//                 violator test of each bank (a pass over its slots), the
//                 shared decision through LDS, and on a taken step the
//                 release, the exact density maintenance and the new state
//   k_seq_commit  the K/V rows of the slots that ended with a candidate
//
// Weights are the binary32 chain of the rest of the update on exact grid
// distances (d2 = |a|^2 + |b|^2 - 2 <a, b>, exact in fp32 for keys on the
// 1/64 grid), so every decision is the one the default stages would take on
// the same pairs.
#include <hip/hip_runtime.h>

#include "dkv_internal.hpp"

namespace dkv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kSeqWaves = 16;  // waves of the k_seq workgroup (banks walked in parallel)

__device__ __forceinline__ uint32_t weight_q(float d2, const Prm &p) {
  return q23_round(pair_weight(d2, p.inv_sigma2, p.p), 8388608.0f);
}

// Register q of a 32 x 32 MFMA tile holds column 8 (q / 4) + 4 h + q % 4.
__device__ __forceinline__ int tile_col(int q, int h) { return 8 * (q >> 2) + 4 * h + (q & 3); }

// ---------------------------------------------------------------------------
// k_seq_gram: workgroup = 4 waves = 32 row items x 128 column items.
// Item u < Mcap is bank slot u (live while u < m), item Mcap + x candidate x.
// Dead items read a live row of the bank array (finite or not, their
// products only reach outputs that are not stored).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void k_seq_gram(dkv_bank bank, dkv_segment seg, Geom g, Prm p, Workspace ws) {
  constexpr int KS = D / 16;
  const int b = blockIdx.z;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const int L = ws.gram_ld, Mcap = g.Mcap, m = ws.m[b];
  auto live = [&](int u) { return u < Mcap ? u < m : u < Mcap + g.N; };
  auto any_live = [&](int u0) {  // items [u0, u0 + 32)
    const int u1 = u0 + 32;
    return (u0 < m) || (u1 > Mcap && u0 < Mcap + g.N);
  };
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 128 + wave * 32;
  if (!any_live(r0) || !any_live(c0) || c0 >= L) return;  // whole wave (no barrier in this kernel)
  const uint16_t *bk = static_cast<const uint16_t *>(bank.k);
  const uint16_t *ck = static_cast<const uint16_t *>(seg.k);
  auto row_ptr = [&](int u) -> const uint16_t * {
    if (u >= Mcap && u < Mcap + g.N) return ck + ((size_t)b * g.N + (u - Mcap)) * D;
    return bk + ((size_t)b * Mcap + (u < Mcap ? u : 0)) * D;
  };
  auto norm_of = [&](int u) -> float {
    if (u >= Mcap && u < Mcap + g.N) return ws.cnorm[(size_t)b * g.N + (u - Mcap)];
    return u < m ? bank.knorm[(size_t)b * Mcap + u] : 0.0f;
  };
  const int ru = r0 + n, cu = c0 + n;  // this lane's row item (B operand) and column item (A operand)
  const uint16_t *rp = row_ptr(ru), *cp = row_ptr(cu);
  f32x16 acc = {};
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    const u32x4 a = *reinterpret_cast<const u32x4 *>(cp + 16 * kk + 8 * h);
    const u32x4 bb = *reinterpret_cast<const u32x4 *>(rp + 16 * kk + 8 * h);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, bb), acc,
                                                  0, 0, 0);
  }
  const float nr = norm_of(ru), nc = norm_of(cu);
  float ncm[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) ncm[q] = __shfl(nc, tile_col(q, h), 32);  // column item's norm (lane cm of this half)
  if (!live(ru)) return;
  uint32_t *row = ws.gram + ((size_t)b * L + ru) * L;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int u = c0 + tile_col(q, h);
    if (u < L && live(u)) row[u] = weight_q((nr + ncm[q]) - 2.0f * acc[q], p);
  }
}

// Lexicographic maximum over the wave of (rt, -prov, -slot): the densest state,
// ties to the smaller provenance, then the lower slot.
struct Best {
  int64_t rt, prov;
  int slot;
};
__device__ __forceinline__ bool better(const Best &a, const Best &b) {
  if (a.rt != b.rt) return a.rt > b.rt;
  if (a.prov != b.prov) return a.prov < b.prov;
  return a.slot < b.slot;
}
__device__ __forceinline__ int64_t shfl_xor_i64(int64_t v, int mask) {
  const uint32_t lo = __shfl_xor((uint32_t)v, mask, 64), hi = __shfl_xor((uint32_t)((uint64_t)v >> 32), mask, 64);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ Best wave_best(Best v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    Best w{shfl_xor_i64(v.rt, o), shfl_xor_i64(v.prov, o), __shfl_xor(v.slot, o, 64)};
    if (better(w, v)) v = w;
  }
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += shfl_xor_i64(v, o);
  return v;
}

// ---------------------------------------------------------------------------
// k_seq: the steps of one group.  Per bank, a slot's state lives in the bank
// arrays (rho, base, prov, knorm) and in ws.grow / ws.lim; every slot is read
// and written by the same lane (slot % 64) of the bank's wave, and a wave
// fences its memory operations at the end of each step.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64 * kSeqWaves) void k_seq(dkv_bank bank, Geom g, Prm p, Workspace ws,
                                                       dkv_update_out out) {
  const int grp = blockIdx.x, nw = blockDim.x >> 6;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int L = ws.gram_ld, Mcap = g.Mcap, N = g.N;
  __shared__ int mcur[kSeqMaxGroup], m0s[kSeqMaxGroup];
  __shared__ int dec_cnt[kSeqMaxGroup], dec_v[kSeqMaxGroup], dec_best[kSeqMaxGroup];
  __shared__ int flag[2][kSeqWaves];
  __shared__ int any_live;
  int steps_taken = 0;
  if (threadIdx.x == 0) any_live = 0;
  __syncthreads();
  // ---- set-up: per-slot items and limits; empty banks take the empty-bank rule
  for (int hh = wave; hh < g.gs; hh += nw) {
    const int b = grp * g.gs + hh;
    const size_t rb = (size_t)b * Mcap;
    const int m0 = ws.m[b];
    const int M = ws.M[b];
    if (l == 0) m0s[hh] = m0;
    if (m0 > 0 && l == 0) any_live = 1;
    if (m0 > 0) {
      for (int s = l; s < m0; s += 64) {
        ws.grow[rb + s] = s;
        ws.lim[rb + s] = ((int64_t)p.tau_num * bank.base[rb + s] + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
      }
      if (l == 0) mcur[hh] = m0;
    } else {
      // the first min(N, M) candidates in source order, densities over that bank (Alg. 1, first branch)
      const int na = min(N, M);
      for (int x = 0; x < na; ++x) {
        const uint32_t *wr = ws.gram + ((size_t)b * L + Mcap + x) * L + Mcap;
        int64_t acc = 0;
        for (int y = l; y < na; y += 64)
          if (y != x) acc += wr[y];
        acc = wave_sum_i64(acc);
        if (l == (x & 63)) {
          bank.rho[rb + x] = acc;
          const int64_t bs = acc > p.delta_q ? acc : p.delta_q;
          bank.base[rb + x] = bs;
          ws.lim[rb + x] = ((int64_t)p.tau_num * bs + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
          ws.grow[rb + x] = Mcap + x;
          bank.prov[rb + x] = ((int64_t)p.block_id << 32) | (int64_t)x;
          bank.knorm[rb + x] = ws.cnorm[(size_t)b * N + x];
        }
      }
      if (l == 0) mcur[hh] = na;
    }
  }
  __threadfence_block();
  __syncthreads();
  // ---- the steps (none when every bank of the group started empty)
  const int nsteps = any_live ? N : 0;
  for (int j = 0; j < nsteps; ++j) {
    int ok_wave = 1;
    for (int hh = wave; hh < g.gs; hh += nw) {
      if (m0s[hh] == 0) continue;  // empty at the start: not part of the shared test
      const int b = grp * g.gs + hh;
      const size_t rb = (size_t)b * Mcap;
      const int m = mcur[hh];
      const int x = ws.order[(size_t)b * N + j];
      const uint32_t *wx = ws.gram + ((size_t)b * L + Mcap + x) * L;
      int cnt = 0, vmin = INT_MAX;
      Best best{INT64_MIN, INT64_MAX, INT_MAX};
      for (int s = l; s < m; s += 64) {
        const int64_t rt = bank.rho[rb + s] + (int64_t)wx[ws.grow[rb + s]];
        if (rt >= ws.lim[rb + s]) {
          ++cnt;
          vmin = min(vmin, s);
        }
        const Best c{rt, bank.prov[rb + s], s};
        if (better(c, best)) best = c;
      }
      cnt = wave_sum_i(cnt);
      vmin = wave_min_i(vmin);
      best = wave_best(best);
      const int e = m + 1 > ws.M[b] ? 1 : 0;
      if (l == 0) {
        dec_cnt[hh] = cnt;
        dec_v[hh] = vmin;
        dec_best[hh] = best.slot;
      }
      ok_wave &= cnt <= e ? 1 : 0;
    }
    if (l == 0) flag[j & 1][wave] = ok_wave;
    __syncthreads();
    int admit = 1;
    for (int w = 0; w < nw; ++w) admit &= flag[j & 1][w];
    if (!admit) continue;
    ++steps_taken;
    for (int hh = wave; hh < g.gs; hh += nw) {
      if (m0s[hh] == 0) continue;
      const int b = grp * g.gs + hh;
      const size_t rb = (size_t)b * Mcap;
      const int m = mcur[hh];
      const int x = ws.order[(size_t)b * N + j];
      const int e = m + 1 > ws.M[b] ? 1 : 0;
      const int ev = dec_cnt[hh] > 0 ? dec_v[hh] : (e ? dec_best[hh] : -1);
      const uint32_t *wx = ws.gram + ((size_t)b * L + Mcap + x) * L;
      const uint32_t *wev = ev >= 0 ? ws.gram + ((size_t)b * L + ws.grow[rb + ev]) * L : nullptr;
      int64_t sum = 0;
      for (int s = l; s < m; s += 64) {
        if (s == ev) continue;
        const int gsl = ws.grow[rb + s];
        const int64_t w = (int64_t)wx[gsl];
        bank.rho[rb + s] += w - (wev ? (int64_t)wev[gsl] : 0);
        sum += w;
      }
      sum = wave_sum_i64(sum);
      const int t = ev >= 0 ? ev : m;
      if (l == (t & 63)) {
        bank.rho[rb + t] = sum;
        const int64_t bs = sum > p.delta_q ? sum : p.delta_q;
        bank.base[rb + t] = bs;
        ws.lim[rb + t] = ((int64_t)p.tau_num * bs + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
        ws.grow[rb + t] = Mcap + x;
        bank.prov[rb + t] = ((int64_t)p.block_id << 32) | (int64_t)x;
        bank.knorm[rb + t] = ws.cnorm[(size_t)b * N + x];
      }
      if (l == 0 && ev < 0) mcur[hh] = m + 1;
    }
    __threadfence_block();
  }
  // ---- results
  if (threadIdx.x == 0 && out.r_star) out.r_star[grp] = steps_taken;
  for (int hh = wave; hh < g.gs; hh += nw) {
    const int b = grp * g.gs + hh;
    const size_t rb = (size_t)b * Mcap, nb = (size_t)b * N;
    const int m = mcur[hh], m0 = m0s[hh];
    if (l == 0) bank.occupancy[b] = m;
    if (p.flags & DKV_POLICY_REFRESH_BASE)
      for (int s = l; s < m; s += 64) {
        const int64_t r = bank.rho[rb + s];
        bank.base[rb + s] = r > p.delta_q ? r : p.delta_q;
      }
    // this block's candidates in the final bank, ascending source index
    for (int x = l; x < N; x += 64) ws.rank[nb + x] = 0;
    __threadfence_block();
    for (int s = l; s < m; s += 64) {
      const int gsl = ws.grow[rb + s];
      if (gsl >= Mcap) ws.rank[nb + (gsl - Mcap)] = 1;
    }
    __threadfence_block();
    int na = 0;
    for (int x0 = 0; x0 < N; x0 += 64) {
      const int x = x0 + l;
      const bool in = x < N && ws.rank[nb + x] != 0;
      const unsigned long long bal = __ballot(in);
      if (in && out.admitted) out.admitted[nb + na + __popcll(bal & ((1ull << l) - 1))] = x;
      na += __popcll(bal);
    }
    if (out.admitted)
      for (int x = na + l; x < N; x += 64) out.admitted[nb + x] = -1;
    // pre-update slots whose state left, ascending
    int nv = 0;
    for (int s0 = 0; s0 < m0; s0 += 64) {
      const int s = s0 + l;
      const bool gone = s < m0 && ws.grow[rb + s] != s;
      const unsigned long long bal = __ballot(gone);
      if (gone && out.evicted) out.evicted[rb + nv + __popcll(bal & ((1ull << l) - 1))] = s;
      nv += __popcll(bal);
    }
    if (out.evicted)
      for (int s = nv + l; s < Mcap; s += 64) out.evicted[rb + s] = -1;
    if (l == 0) {
      if (out.n_admitted) out.n_admitted[b] = na;
      if (out.n_evicted) out.n_evicted[b] = nv;
    }
  }
}

// ---------------------------------------------------------------------------
// k_seq_commit: K and V rows of every slot whose final state is a candidate,
// one 16-byte chunk per thread (a key row and its value row per 2 * D / 8 lanes).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void k_seq_commit(dkv_bank bank, dkv_segment seg, Geom g, Workspace ws) {
  constexpr int CH = D / 8;             // 16-byte chunks per bf16 row
  constexpr int kSlots = 256 / (2 * CH);  // slots per workgroup
  const int b = blockIdx.y;
  const int s = blockIdx.x * kSlots + threadIdx.x / (2 * CH);
  const int c = threadIdx.x % (2 * CH);
  const int m = bank.occupancy[b];
  if (s >= m) return;
  const size_t rb = (size_t)b * g.Mcap;
  const int gsl = ws.grow[rb + s];
  if (gsl < g.Mcap) return;
  const int x = gsl - g.Mcap;
  const bool isv = c >= CH;
  const int cc = isv ? c - CH : c;
  const uint16_t *src = static_cast<const uint16_t *>(isv ? seg.v : seg.k) + ((size_t)b * g.N + x) * D;
  uint16_t *dst = static_cast<uint16_t *>(isv ? bank.v : bank.k) + (rb + s) * D;
  reinterpret_cast<u32x4 *>(dst)[cc] = reinterpret_cast<const u32x4 *>(src)[cc];
}

template <int D>
hipError_t seq_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                    const dkv_update_out &out, const Workspace &ws, hipStream_t s) {
  const int L = ws.gram_ld;
  if (L > 0 && g.N > 0) {
    const dim3 grid((unsigned)((L + 127) / 128), (unsigned)((L + 31) / 32), (unsigned)g.B);
    k_seq_gram<D><<<grid, 256, 0, s>>>(bank, seg, g, p, ws);
  }
  const int waves = g.gs < kSeqWaves ? g.gs : kSeqWaves;
  k_seq<<<g.G, 64 * waves, 0, s>>>(bank, g, p, ws, out);
  if (g.N > 0) {
    constexpr int kSlots = 256 / (2 * (D / 8));
    k_seq_commit<D><<<dim3((unsigned)((g.Mcap + kSlots - 1) / kSlots), (unsigned)g.B), 256, 0, s>>>(bank, seg, g,
                                                                                                  ws);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sequential(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                             const dkv_update_out &out, const Workspace &ws, hipStream_t s) {
  if (g.d == 128) return seq_impl<128>(bank, seg, g, p, out, ws, s);
  return seq_impl<64>(bank, seg, g, p, out, ws, s);
}

}  // namespace dkv
