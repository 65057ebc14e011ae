// Within-block sequential competition (Supp. E, "Within-block competition";
// DKV_POLICY_SEQUENTIAL in include/densitykv.h): the candidates of a block are
// offered one at a time, in the order fixed at the start of the block, and
// every step is decided against the banks as the earlier steps left them.
//
// The groups run in batches of whole groups (as many as the workspace's
// weight area holds); per batch:
//   k_seq_gram    W between every pair of items of a bank, the items being its
//                 slots 0..Mcap-1 (pre-update states) and its candidates, on
//                 bf16 MFMA (32 x 32 tiles), stored as [batch banks, L, L]
//                 uint32 with L = Mcap + N
//   k_seq_setup   per bank, in the workspace: slot items and violation
//                 limits, or the items of the empty-bank rule for a bank that
//                 starts empty
//   k_seq_coop    the steps, several workgroups per group (cooperative
//                 launch): each holds up to 2,048 slots of one bank in
//                 registers; per step the one-candidate violator test of its
//                 slots, one record per workgroup exchanged through global
//                 memory, the shared decision, and on a taken step the
//                 release, the exact density maintenance and the new state
//   k_seq_results per bank: the states of a bank that started empty,
//                 refreshed baselines, admitted and released lists
//   k_seq         the same steps in one workgroup per group (one wave per
//                 bank, the state in the bank arrays), for groups the
//                 cooperative walk does not take
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

// Pairwise weights of bank b, one of the banks of the batch being walked.
__device__ __forceinline__ const uint32_t *bank_gram(const Workspace &ws, int b) {
  const size_t L = (size_t)ws.gram_ld;
  return ws.gram + (size_t)(b - ws.seq_b0) * L * L;
}

// ---------------------------------------------------------------------------
// k_seq_gram: workgroup = 4 waves = 32 row items x kGramCols column items; a
// wave keeps its 32 row keys (the B operand) in registers and walks
// kGramCols / 128 tiles of 32 columns.  Item u < Mcap is bank slot u (live
// while u < m), item Mcap + x candidate x.  Dead items read a live row of the
// bank array (finite or not, their products only reach outputs that are not
// stored).
// ---------------------------------------------------------------------------
constexpr int kGramCols = 512;

template <int D>
__global__ __launch_bounds__(256) void k_seq_gram(dkv_bank bank, dkv_segment seg, Geom g, Prm p, Workspace ws) {
  constexpr int KS = D / 16;
  const int b = ws.seq_b0 + (int)blockIdx.z;  // bank blockIdx.z of the batch
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const int L = ws.gram_ld, Mcap = g.Mcap, m = ws.m[b];
  auto live = [&](int u) { return u < Mcap ? u < m : u < Mcap + g.N; };
  auto any_live = [&](int u0) {  // items [u0, u0 + 32)
    const int u1 = u0 + 32;
    return (u0 < m) || (u1 > Mcap && u0 < Mcap + g.N);
  };
  const int r0 = blockIdx.y * 32;
  if (!any_live(r0)) return;  // whole workgroup (no barrier in this kernel)
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
  const int ru = r0 + n;  // this lane's row item (B operand)
  const uint16_t *rp = row_ptr(ru);
  bf16x8 bb[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) bb[kk] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(rp + 16 * kk + 8 * h));
  const float nr = norm_of(ru);
  const bool row_live = live(ru);
  // W is symmetric (the same products summed in the same order, and |a|^2 +
  // |b|^2 commutes), so W(ru, u) is stored at [u][ru]: the 32 lanes of a half
  // write 32 consecutive entries of one row.
  uint32_t *col = ws.gram + (size_t)blockIdx.z * L * L + ru;
  for (int c0 = blockIdx.x * kGramCols + wave * 32; c0 < min(L, (int)(blockIdx.x + 1) * kGramCols); c0 += 128) {
    if (!any_live(c0)) continue;  // uniform over the wave
    const int cu = c0 + n;  // this lane's column item (A operand)
    const uint16_t *cp = row_ptr(cu);
    f32x16 acc = {};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const u32x4 a = *reinterpret_cast<const u32x4 *>(cp + 16 * kk + 8 * h);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), bb[kk], acc, 0, 0, 0);
    }
    const float nc = norm_of(cu);
    float ncm[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) ncm[q] = __shfl(nc, tile_col(q, h), 32);  // column item's norm
    if (row_live) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int u = c0 + tile_col(q, h);
        if (u < L && live(u)) col[(size_t)u * L] = weight_q((nr + ncm[q]) - 2.0f * acc[q], p);
      }
    }
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

__device__ __forceinline__ int64_t lim_of(int64_t base, const Prm &p) {
  return ((int64_t)p.tau_num * base + ((1ll << p.tau_shift) - 1)) >> p.tau_shift;
}

// Set-up of bank b by one wave, in the workspace only: per-slot items and
// limits of a bank that holds states; for a bank that is empty, the items of
// the empty-bank rule (the first min(N, M) candidates in source order; Alg. 1,
// first branch), whose states seq_empty_commit writes.  Returns the occupancy
// the steps start from.
__device__ int seq_setup_bank(const dkv_bank &bank, const Geom &g, const Prm &p, const Workspace &ws, int b, int l) {
  const int Mcap = g.Mcap, N = g.N;
  const size_t rb = (size_t)b * Mcap;
  const int m0 = ws.m[b];
  if (m0 > 0) {
    for (int s = l; s < m0; s += 64) {
      ws.grow[rb + s] = s;
      ws.lim[rb + s] = lim_of(bank.base[rb + s], p);
    }
    return m0;
  }
  const int na = min(N, ws.M[b]);
  for (int x = l; x < na; x += 64) ws.grow[rb + x] = Mcap + x;
  return na;
}

// The states of a bank that was empty at the start of the block (the
// empty-bank rule): slot x holds candidate x, its density the sum of its
// weights to the other admitted candidates.  One wave.
__device__ void seq_empty_commit(const dkv_bank &bank, const Geom &g, const Prm &p, const Workspace &ws, int b,
                                 int l) {
  const int L = ws.gram_ld, Mcap = g.Mcap, N = g.N;
  const size_t rb = (size_t)b * Mcap;
  const int na = min(N, ws.M[b]);
  const uint32_t *gb = bank_gram(ws, b);
  for (int x = 0; x < na; ++x) {
    const uint32_t *wr = gb + (size_t)(Mcap + x) * L + Mcap;
    int64_t acc = 0;
    for (int y = l; y < na; y += 64)
      if (y != x) acc += wr[y];
    acc = wave_sum_i64(acc);
    if (l == (x & 63)) {
      bank.rho[rb + x] = acc;
      bank.base[rb + x] = acc > p.delta_q ? acc : p.delta_q;
      bank.prov[rb + x] = ((int64_t)p.block_id << 32) | (int64_t)x;
      bank.knorm[rb + x] = ws.cnorm[(size_t)b * N + x];
    }
  }
}

// Results of bank b by one wave, from its final occupancy m and the occupancy
// m0 it held before the update: refreshed baselines, the admitted candidates
// (ascending source index) and the pre-update slots whose state left.
__device__ void seq_results_bank(const dkv_bank &bank, const Geom &g, const Prm &p, const Workspace &ws,
                                 const dkv_update_out &out, int b, int l, int m, int m0) {
  const int Mcap = g.Mcap, N = g.N;
  const size_t rb = (size_t)b * Mcap, nb = (size_t)b * N;
  if (l == 0) bank.occupancy[b] = m;
  if (p.flags & DKV_POLICY_REFRESH_BASE)
    for (int s = l; s < m; s += 64) {
      const int64_t r = bank.rho[rb + s];
      bank.base[rb + s] = r > p.delta_q ? r : p.delta_q;
    }
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

// ---------------------------------------------------------------------------
// k_seq: the steps of one group in one workgroup (any bank size).  Per bank, a
// slot's state lives in the bank arrays (rho, base, prov, knorm) and in
// ws.grow / ws.lim; every slot is read and written by the same lane
// (slot % 64) of the bank's wave, and a wave fences its memory operations at
// the end of each step.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64 * kSeqWaves) void k_seq(dkv_bank bank, Geom g, Prm p, Workspace ws,
                                                       dkv_update_out out) {
  const int grp = ws.seq_b0 / g.gs + (int)blockIdx.x, nw = blockDim.x >> 6;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int L = ws.gram_ld, Mcap = g.Mcap, N = g.N;
  __shared__ int mcur[kSeqMaxGroup], m0s[kSeqMaxGroup];
  __shared__ int dec_cnt[kSeqMaxGroup], dec_v[kSeqMaxGroup], dec_best[kSeqMaxGroup];
  __shared__ int flag[2][kSeqWaves];
  __shared__ int any_live;
  int steps_taken = 0;
  if (threadIdx.x == 0) any_live = 0;
  __syncthreads();
  for (int hh = wave; hh < g.gs; hh += nw) {
    const int b = grp * g.gs + hh;
    const int m0 = ws.m[b];
    const int mc = seq_setup_bank(bank, g, p, ws, b, l);
    if (m0 == 0) seq_empty_commit(bank, g, p, ws, b, l);
    if (l == 0) {
      m0s[hh] = m0;
      mcur[hh] = mc;
      if (m0 > 0) any_live = 1;
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
      const uint32_t *wx = bank_gram(ws, b) + (size_t)(Mcap + x) * L;
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
      const uint32_t *wx = bank_gram(ws, b) + (size_t)(Mcap + x) * L;
      const uint32_t *wev = ev >= 0 ? bank_gram(ws, b) + (size_t)ws.grow[rb + ev] * L : nullptr;
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
        ws.lim[rb + t] = lim_of(bs, p);
        ws.grow[rb + t] = Mcap + x;
        bank.prov[rb + t] = ((int64_t)p.block_id << 32) | (int64_t)x;
        bank.knorm[rb + t] = ws.cnorm[(size_t)b * N + x];
      }
      if (l == 0 && ev < 0) mcur[hh] = m + 1;
    }
    __threadfence_block();
  }
  if (threadIdx.x == 0 && out.r_star) out.r_star[grp] = steps_taken;
  for (int hh = wave; hh < g.gs; hh += nw)
    seq_results_bank(bank, g, p, ws, out, grp * g.gs + hh, l, mcur[hh], m0s[hh]);
}

// ---------------------------------------------------------------------------
// Multi-workgroup walk.  Workgroup (b, q) of a bank holds the slots
// q * 256 S + k * 256 + thread (k < S, S = 8 or 16) in registers: rho, limit,
// item and provenance.  Per step every workgroup posts one record (its
// violator count, its first violator, its densest state and the sum of its
// weights to the candidate) to global memory as step-tagged words; wave 0 of
// every workgroup polls the group's records until they carry the step's tag
// and takes the shared decision from them.  The weights to the next
// candidate are gathered while the records are exchanged.  Launched
// cooperatively, so all workgroups of the grid are resident together and
// every wait ends; a wait that still exceeds kSpinCap polls ends the walk
// with r_star = -1.
// ---------------------------------------------------------------------------
constexpr int kCoopThreads = 256;  // threads of a workgroup of the walk
constexpr int kCoopWaves = kCoopThreads / 64;
// slots per thread: 8 (2,048 per workgroup), or 16 when a group would need
// more than kSeqMaxMembers workgroups of 2,048 slots
constexpr int kSpinCap = 1 << 22;

// record words: 0 cnt | e << 32, 1 vmin | W(vmin) << 32, 2 item(vmin) | best slot << 32,
// 3 W(best) | item(best) << 32, 4 best rt, 5 best prov, 6 sum of W
struct Rec {
  int cnt, e, vmin, best_slot;
  uint32_t wv, gv, wb, gb;
  int64_t rt, prov, total;
};
__device__ __forceinline__ void rec_merge(Rec &a, const Rec &o) {
  a.cnt += o.cnt;
  a.total += o.total;
  if (o.vmin < a.vmin) {
    a.vmin = o.vmin;
    a.wv = o.wv;
    a.gv = o.gv;
  }
  if (better(Best{o.rt, o.prov, o.best_slot}, Best{a.rt, a.prov, a.best_slot})) {
    a.rt = o.rt;
    a.prov = o.prov;
    a.best_slot = o.best_slot;
    a.wb = o.wb;
    a.gb = o.gb;
  }
}
__device__ __forceinline__ Rec rec_shfl(const Rec &r, int src) {
  auto sh64 = [&](int64_t v) {
    const uint32_t lo = __shfl((uint32_t)v, src, 64), hi = __shfl((uint32_t)((uint64_t)v >> 32), src, 64);
    return (int64_t)(((uint64_t)hi << 32) | lo);
  };
  Rec o;
  o.cnt = __shfl(r.cnt, src, 64);
  o.e = __shfl(r.e, src, 64);
  o.vmin = __shfl(r.vmin, src, 64);
  o.best_slot = __shfl(r.best_slot, src, 64);
  o.wv = __shfl(r.wv, src, 64);
  o.gv = __shfl(r.gv, src, 64);
  o.wb = __shfl(r.wb, src, 64);
  o.gb = __shfl(r.gb, src, 64);
  o.rt = sh64(r.rt);
  o.prov = sh64(r.prov);
  o.total = sh64(r.total);
  return o;
}
// Wave reduction of the lanes' records.  The count rides in the bits from 40
// up of the weight sum (a wave holds at most 64 x 16 = 1,024 slots, so its sum
// of weights <= 2^23 stays at or below 2^33, under bit 40),
// the slots and the densest state's key are reduced level by level, and the
// weights and items of the first violator and of the densest state are then
// read once from the lanes that hold them (a slot belongs to one lane).
__device__ __forceinline__ Rec rec_wave(const Rec &r) {
  int64_t sc = r.total + ((int64_t)r.cnt << 40);
  int vmin = r.vmin;
  Best best{r.rt, r.prov, r.best_slot};
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    sc += shfl_xor_i64(sc, o);
    vmin = min(vmin, __shfl_xor(vmin, o, 64));
    const Best w{shfl_xor_i64(best.rt, o), shfl_xor_i64(best.prov, o), __shfl_xor(best.slot, o, 64)};
    if (better(w, best)) best = w;
  }
  Rec w{(int)(sc >> 40), r.e, vmin, best.slot, 0u, 0u, 0u, 0u, best.rt, best.prov, sc & ((1ll << 40) - 1)};
  const unsigned long long hv = __ballot(vmin != INT_MAX && r.vmin == vmin);
  const unsigned long long hb = __ballot(best.slot != INT_MAX && r.best_slot == best.slot);
  const int lv = hv ? __ffsll((long long)hv) - 1 : 0, lb = hb ? __ffsll((long long)hb) - 1 : 0;
  w.wv = __shfl(r.wv, lv, 64);
  w.gv = __shfl(r.gv, lv, 64);
  w.wb = __shfl(r.wb, lb, 64);
  w.gb = __shfl(r.gb, lb, 64);
  return w;
}

// A record travels as kRecWords 64-bit words, each with a 48-bit payload and
// the step tag j + 1 in its top 16 bits (N < 2^13): counts, slots (< 2^15,
// 0xFFFF for none) and items (< 2^16) in 16 bits, weights (<= 2^23) in 24,
// densities (< 2^39) in 48, the provenance in two 32-bit halves.  Each word
// is stored and loaded as one relaxed device-scope atomic, so a reader that
// sees the tag in every word has the whole record of that step.
constexpr int kRecWords = 7;
constexpr uint64_t kPayload = (1ull << 48) - 1;
__device__ __forceinline__ uint64_t slot16(int s) { return s == INT_MAX ? 0xFFFFull : (uint64_t)s; }
__device__ __forceinline__ int unslot16(uint64_t v) { return v == 0xFFFFull ? INT_MAX : (int)v; }
__device__ __forceinline__ void rec_encode(const Rec &w, uint64_t *v) {
  v[0] = (uint64_t)w.cnt | slot16(w.vmin) << 16 | slot16(w.best_slot) << 32;
  v[1] = (uint64_t)w.wv | (uint64_t)w.gv << 24 | (uint64_t)w.e << 40;
  v[2] = (uint64_t)w.wb | (uint64_t)w.gb << 24;
  v[3] = w.rt == INT64_MIN ? 0ull : (uint64_t)(w.rt + 1);
  v[4] = (uint64_t)w.prov & 0xFFFFFFFFull;
  v[5] = (uint64_t)w.prov >> 32;
  v[6] = (uint64_t)w.total;
}
__device__ __forceinline__ Rec rec_decode(const uint64_t *v) {
  Rec o;
  o.cnt = (int)(v[0] & 0xFFFF);
  o.vmin = unslot16((v[0] >> 16) & 0xFFFF);
  o.best_slot = unslot16((v[0] >> 32) & 0xFFFF);
  o.wv = (uint32_t)(v[1] & 0xFFFFFF);
  o.gv = (uint32_t)((v[1] >> 24) & 0xFFFF);
  o.e = (int)((v[1] >> 40) & 1);
  o.wb = (uint32_t)(v[2] & 0xFFFFFF);
  o.gb = (uint32_t)((v[2] >> 24) & 0xFFFF);
  const uint64_t r3 = v[3] & kPayload;
  o.rt = r3 == 0 ? INT64_MIN : (int64_t)r3 - 1;
  o.prov = (int64_t)(((v[5] & 0xFFFFFFFFull) << 32) | (v[4] & 0xFFFFFFFFull));
  o.total = (int64_t)(v[6] & kPayload);
  return o;
}

__global__ __launch_bounds__(64 * kSeqWaves) void k_seq_setup(dkv_bank bank, Geom g, Prm p, Workspace ws) {
  const int grp = ws.seq_b0 / g.gs + (int)blockIdx.x, nw = blockDim.x >> 6;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  for (int hh = wave; hh < g.gs; hh += nw) {
    const int b = grp * g.gs + hh;
    const int mc = seq_setup_bank(bank, g, p, ws, b, l);
    if (l == 0) {
      ws.m_new[b] = mc;
      ws.n_ev[b] = 0;  // set to 1 by a workgroup of the bank whose walk timed out
    }
  }
  if (threadIdx.x == 0) ws.r_star[grp] = 0;
  // no record of this call carries a step tag yet
  uint64_t *recs = ws.seq_rec + (size_t)grp * 2 * kSeqMaxMembers * 8;
  for (int i = threadIdx.x; i < 2 * kSeqMaxMembers * 8; i += blockDim.x) recs[i] = 0;
}

template <int S>
__global__ __launch_bounds__(kCoopThreads) void k_seq_coop(dkv_bank bank, Geom g, Prm p, Workspace ws, int P) {
  const int b = ws.seq_b0 + (int)blockIdx.x / P, q = blockIdx.x % P;
  const int grp = b / g.gs, hh = b % g.gs;
  const int tid = threadIdx.x, wave = tid >> 6, l = tid & 63;
  const int L = ws.gram_ld, Mcap = g.Mcap, N = g.N;
  if (ws.m[b] == 0) return;  // empty at the start: the empty-bank rule, outside the walk
  __shared__ Rec red[kCoopWaves];
  __shared__ int dec_admit, dec_ev, dec_gev, dec_stop;
  __shared__ int64_t dec_sum;
  const size_t rb = (size_t)b * Mcap, nb = (size_t)b * N;
  constexpr int kSlotsWg = kCoopThreads * S;  // slots per workgroup
  const int s0 = q * kSlotsWg;
  const int nmem = g.gs * P;
  // wave 0, lane l reads the record of member l = (head l / P, part l % P)
  const bool lane_live = l < nmem && ws.m[grp * g.gs + l / P] > 0;
  int m = ws.m_new[b];
  const int M = ws.M[b];
  const uint32_t *gb = bank_gram(ws, b);
  int64_t rho[S], lim[S], prov[S];
  int item[S];
  uint32_t wn[S];
#pragma unroll
  for (int k = 0; k < S; ++k) {
    const int s = s0 + k * kCoopThreads + tid;
    const bool lv = s < m;
    rho[k] = lv ? bank.rho[rb + s] : 0;
    lim[k] = lv ? ws.lim[rb + s] : 0;
    prov[k] = lv ? bank.prov[rb + s] : 0;
    item[k] = lv ? ws.grow[rb + s] : 0;
  }
  int x_next = ws.order[nb];
  {
    const uint32_t *row = gb + (size_t)(Mcap + x_next) * L;
#pragma unroll
    for (int k = 0; k < S; ++k) wn[k] = s0 + k * kCoopThreads + tid < m ? row[item[k]] : 0u;
  }
  int steps_taken = 0, stop = 0;
  uint64_t *recs = ws.seq_rec + (size_t)grp * 2 * kSeqMaxMembers * 8;
  for (int j = 0; j < N && !stop; ++j) {
    const int x = x_next;
    if (j + 1 < N) x_next = ws.order[nb + j + 1];
    uint32_t wx[S];
    // ---- test of this workgroup's slots against candidate x
    Rec r{0, m + 1 > M ? 1 : 0, INT_MAX, INT_MAX, 0u, 0u, 0u, 0u, INT64_MIN, INT64_MAX, 0};
#pragma unroll
    for (int k = 0; k < S; ++k) {
      wx[k] = wn[k];
      const int s = s0 + k * kCoopThreads + tid;
      if (s < m) {
        const int64_t rt = rho[k] + (int64_t)wx[k];
        if (rt >= lim[k]) {
          ++r.cnt;
          if (s < r.vmin) {
            r.vmin = s;
            r.wv = wx[k];
            r.gv = (uint32_t)item[k];
          }
        }
        if (better(Best{rt, prov[k], s}, Best{r.rt, r.prov, r.best_slot})) {
          r.rt = rt;
          r.prov = prov[k];
          r.best_slot = s;
          r.wb = wx[k];
          r.gb = (uint32_t)item[k];
        }
        r.total += wx[k];
      }
    }
    r = rec_wave(r);
    if (l == 0) red[wave] = r;
    __syncthreads();
    if (tid == 0 && nmem > 1) {
      Rec w = red[0];
#pragma unroll
      for (int v = 1; v < kCoopWaves; ++v) rec_merge(w, red[v]);
      uint64_t v[kRecWords];
      rec_encode(w, v);
      uint64_t *dst = recs + ((size_t)(j & 1) * kSeqMaxMembers + hh * P + q) * 8;
      const uint64_t tag = (uint64_t)(j + 1) << 48;
#pragma unroll
      for (int i = 0; i < kRecWords; ++i)
        __hip_atomic_store(dst + i, v[i] | tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // ---- gather the weights to the next candidate while the records travel
    if (j + 1 < N) {
      const uint32_t *row = gb + (size_t)(Mcap + x_next) * L;
#pragma unroll
      for (int k = 0; k < S; ++k) wn[k] = s0 + k * kCoopThreads + tid < m ? row[item[k]] : 0u;
    }
    if (wave == 0) {
      Rec o{0, 0, INT_MAX, INT_MAX, 0u, 0u, 0u, 0u, INT64_MIN, INT64_MAX, 0};
      int polls = 0;
      if (nmem == 1) {
        // a single workgroup in the group: its own record is the decision's input
        if (l == 0) {
          o = red[0];
#pragma unroll
          for (int v = 1; v < kCoopWaves; ++v) rec_merge(o, red[v]);
        }
      } else if (lane_live) {
        // poll until every word of member l's record carries this step's tag
        const uint64_t *src = recs + ((size_t)(j & 1) * kSeqMaxMembers + l) * 8;
        const uint64_t tag = (uint64_t)(j + 1);
        uint64_t v[kRecWords];
        for (;;) {
          bool ready = true;
#pragma unroll
          for (int i = 0; i < kRecWords; ++i) {
            v[i] = __hip_atomic_load(src + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ready &= (v[i] >> 48) == tag;
          }
          if (ready || ++polls >= kSpinCap) break;
          __builtin_amdgcn_s_sleep(1);
        }
        if (polls < kSpinCap) o = rec_decode(v);
      }
      const int timed_out = __ballot(polls >= kSpinCap) != 0ull ? 1 : 0;
      // merge the parts of each bank into its first part's lane
      for (int i = 1; i < P; ++i) {
        const Rec v = rec_shfl(o, l + i < 64 ? l + i : l);
        if (l % P == 0 && l + i < nmem) rec_merge(o, v);
      }
      const bool lead = l % P == 0 && lane_live;
      const unsigned long long bad = __ballot(lead && o.cnt > o.e);
      const Rec own = rec_shfl(o, hh * P);
      if (l == 0) {
        const int admit = bad == 0ull ? 1 : 0;
        const int ev = own.cnt > 0 ? own.vmin : (own.e ? own.best_slot : -1);
        dec_admit = admit;
        dec_ev = ev;
        dec_gev = (int)(own.cnt > 0 ? own.gv : own.gb);
        dec_sum = own.total - (ev >= 0 ? (int64_t)(own.cnt > 0 ? own.wv : own.wb) : 0);
        dec_stop = timed_out;
      }
    }
    __syncthreads();
    stop = dec_stop;
    if (stop || !dec_admit) continue;
    ++steps_taken;
    const int ev = dec_ev;
    if (ev >= 0) {
      const uint32_t *row = gb + (size_t)dec_gev * L;
#pragma unroll
      for (int k = 0; k < S; ++k) {
        const int s = s0 + k * kCoopThreads + tid;
        if (s < m && s != ev) rho[k] += (int64_t)wx[k] - (int64_t)row[item[k]];
      }
    } else {
#pragma unroll
      for (int k = 0; k < S; ++k)
        if (s0 + k * kCoopThreads + tid < m) rho[k] += (int64_t)wx[k];
    }
    const int t = ev >= 0 ? ev : m;
    const int tl = t - s0;
    if (tl >= 0 && tl < kSlotsWg && tl % kCoopThreads == tid) {
      const int kt = tl / kCoopThreads;
      const int64_t sum = dec_sum;
      const int64_t bs = sum > p.delta_q ? sum : p.delta_q;
      const uint32_t wnew = j + 1 < N ? gb[(size_t)(Mcap + x_next) * L + Mcap + x] : 0u;
#pragma unroll
      for (int k = 0; k < S; ++k)
        if (k == kt) {
          rho[k] = sum;
          lim[k] = lim_of(bs, p);
          item[k] = Mcap + x;
          prov[k] = ((int64_t)p.block_id << 32) | (int64_t)x;
          wn[k] = wnew;
        }
      bank.base[rb + t] = bs;
      bank.prov[rb + t] = ((int64_t)p.block_id << 32) | (int64_t)x;
      bank.knorm[rb + t] = ws.cnorm[nb + x];
    }
    if (ev < 0) ++m;
  }
#pragma unroll
  for (int k = 0; k < S; ++k) {
    const int s = s0 + k * kCoopThreads + tid;
    if (s < m) {
      bank.rho[rb + s] = rho[k];
      ws.grow[rb + s] = item[k];
    }
  }
  if (tid == 0 && stop) ws.n_ev[b] = 1;
  if (q == 0 && tid == 0) {
    ws.m_new[b] = m;
    atomicMax(ws.r_star + grp, steps_taken);  // equal in every workgroup of the group
  }
}

__global__ __launch_bounds__(64 * kSeqWaves) void k_seq_results(dkv_bank bank, Geom g, Prm p, Workspace ws,
                                                               dkv_update_out out) {
  const int grp = ws.seq_b0 / g.gs + (int)blockIdx.x, nw = blockDim.x >> 6;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  if (threadIdx.x == 0 && out.r_star) {
    int timed_out = 0;
    for (int h2 = 0; h2 < g.gs; ++h2) timed_out |= ws.n_ev[grp * g.gs + h2];
    out.r_star[grp] = timed_out ? -1 : ws.r_star[grp];
  }
  for (int hh = wave; hh < g.gs; hh += nw) {
    const int b = grp * g.gs + hh;
    if (ws.m[b] == 0) seq_empty_commit(bank, g, p, ws, b, l);
    seq_results_bank(bank, g, p, ws, out, b, l, ws.m_new[b], ws.m[b]);
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
  const int b = ws.seq_b0 + (int)blockIdx.y;
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

// Whether a cooperative launch of nblocks k_seq_coop<S> workgroups fits the
// current device (all of them resident at once).
template <int S>
bool coop_fits(int nblocks) {
  int dev = 0, coop = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop) return false;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return false;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_seq_coop<S>, kCoopThreads, 0) != hipSuccess) return false;
  return (long)per_cu * cus >= nblocks;
}

template <int D>
hipError_t seq_impl(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                    const dkv_update_out &out, const Workspace &ws, hipStream_t s) {
  const int L = ws.gram_ld;
  const int waves = g.gs < kSeqWaves ? g.gs : kSeqWaves;
  // the groups run in batches of ws.seq_groups (their pairwise weights fill the area)
  if (ws.seq_groups < 1) return hipErrorInvalidValue;
  const int per_batch = ws.seq_groups * g.gs;   // banks
  // workgroups per bank with 8 and with 16 slots per thread
  int P8 = (g.Mcap + 8 * kCoopThreads - 1) / (8 * kCoopThreads);
  int P16 = (g.Mcap + 16 * kCoopThreads - 1) / (16 * kCoopThreads);
  // Which walk runs is decided here, before anything is enqueued, for a full
  // batch (a shorter last batch fits when a full one does).
  const int full = per_batch < g.B ? per_batch : g.B;
  const bool use8 = g.N > 0 && g.gs * P8 <= kSeqMaxMembers && coop_fits<8>(full * P8);
  const bool use16 = !use8 && g.N > 0 && g.gs * P16 <= kSeqMaxMembers && coop_fits<16>(full * P16);
  for (int b0 = 0; b0 < g.B; b0 += per_batch) {
    const int nb = per_batch < g.B - b0 ? per_batch : g.B - b0;
    const unsigned ngroups = (unsigned)(nb / g.gs);
    Workspace wb = ws;
    wb.seq_b0 = b0;
    if (L > 0 && g.N > 0) {
      const dim3 grid((unsigned)((L + kGramCols - 1) / kGramCols), (unsigned)((L + 31) / 32), (unsigned)nb);
      k_seq_gram<D><<<grid, 256, 0, s>>>(bank, seg, g, p, wb);
    }
    if (use8 || use16) {
      // the set-up writes the workspace only; the banks change from the walk on
      k_seq_setup<<<ngroups, 64 * waves, 0, s>>>(bank, g, p, wb);
      dkv_bank a_bank = bank;
      Geom a_g = g;
      Prm a_p = p;
      Workspace a_ws = wb;
      int *P = use8 ? &P8 : &P16;
      void *args[] = {&a_bank, &a_g, &a_p, &a_ws, P};
      const void *kern = use8 ? reinterpret_cast<const void *>(k_seq_coop<8>) : reinterpret_cast<const void *>(k_seq_coop<16>);
      const hipError_t e = hipLaunchCooperativeKernel(kern, dim3((unsigned)(nb * *P)), dim3(kCoopThreads), args, 0, s);
      if (e != hipSuccess) return e;
      k_seq_results<<<ngroups, 64 * waves, 0, s>>>(bank, g, p, wb, out);
    } else {
      k_seq<<<ngroups, 64 * waves, 0, s>>>(bank, g, p, wb, out);
    }
    if (g.N > 0) {
      constexpr int kSlots = 256 / (2 * (D / 8));
      k_seq_commit<D><<<dim3((unsigned)((g.Mcap + kSlots - 1) / kSlots), (unsigned)nb), 256, 0, s>>>(bank, seg, g,
                                                                                                   wb);
    }
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
