// Native attention over [retained bank; local window; sink] on gfx950.
//
// out = softmax(q K^T * scale) V with K = [bank k[0:m_b]; window k; sink k],
// the backbone's own attention reading the retained bank together with the
// local window (Sec. 1, Fig. 1; logit of Sec. 3.2) and, in the paper's
// deployment context, a first-frame sink (Supp. D, memory budget and temporal
// alignment).  Every segment is optional.  Online (streaming) softmax in
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
                                                            KvSeg win, KvSeg sink, void *out, float scale_log2,
                                                            Geom g) {
  const int b = blockIdx.y, qi = blockIdx.x * kAThreads + threadIdx.x;
  const bool act = qi < nq;
  const int M = clampi(bank.budget[b], 0, g.Mcap);
  const int m = clampi(bank.occupancy[b], 0, M);
  const int nw = win.n, ns = sink.n;
  const int total = m + nw + ns;
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
        } else if (key < m + nw) {
          const size_t r = ((size_t)b * nw + (key - m)) * D + j;
          kv = load_elem<DT>(win.k, r);
          vv = load_elem<DT>(win.v, r);
        } else {
          const size_t r = ((size_t)b * ns + (key - m - nw)) * D + j;
          kv = load_elem<DT>(sink.k, r);
          vv = load_elem<DT>(sink.v, r);
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
// A workgroup of 8 waves owns 256 queries, 32 per wave.  Per tile of 64 keys:
//   S^T = K Q^T     A = K tile (LDS), B = Q^T (registers): lane l <-> query
//                   l % 32, registers <-> keys, so the softmax row statistics
//                   stay inside the lane (plus one exchange with lane l ^ 32);
//   O^T += V^T P^T  B = P straight from the S registers (bf16); A = V^T read
//                   from the row-major V tile with the transposing LDS read
//                   (ds_read_b64_tr_b16).  Inside each 16-key K step the key
//                   order is permuted identically in both operands
//                   (slot 8h + j <-> key 8 (j / 4) + 4 h + j % 4).
// K and V tiles go global -> LDS with 16-byte buffer loads to LDS (no VGPR
// staging) into a ring of three stages (two tiles in flight while one is
// used); rows are stored with an XOR swizzle of their
// 16-byte chunks so that both the K reads and the transposed V reads are free
// of LDS bank conflicts.  Within a tile the LDS fragment reads are scheduled
// ahead of the MFMAs that use them (6 MFMAs ahead for S, 4 for P V).
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kFWaves = 8;
constexpr int kFQ = 32 * kFWaves;  // queries per workgroup
constexpr int kFK = 64;            // keys per tile
constexpr int kFStages = 3;        // K/V tiles resident in LDS (2 in flight while 1 is used)
// Word 3 of a raw buffer resource: 32-bit data format, no swizzle, no
// thread-id addressing.
constexpr int kBufferRsrcWord3 = 0x00020000;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

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

// The direct-to-LDS loads of one K or V tile.  Lane i of a load writes 16
// bytes at LDS offset 16 i of its 1 KB block, i.e. physical chunk pc of row r;
// it fetches logical chunk swz(r, pc) (the XOR swizzle is an involution, so
// logical chunk c lands at physical swz(r, c)).  These byte offsets within a
// tile are the same for every tile, so they are computed once per lane; the
// tile's first row is the uniform buffer base and the buffer ends after its
// nvalid rows, so the rows beyond read as zero (finite; their scores are
// masked and their weights are 0).  The loads are raw buffer loads to LDS
// rather than global loads to LDS: with a global load to LDS in flight the
// compiler counts every later LDS read as possibly out of order and waits for
// all of them before each use, which serializes the MFMAs on the LDS latency.
template <int D>
struct FTileOff {
  static constexpr int kPerWave = FCfg<D>::kLoadsPerTile / kFWaves;  // loads per wave per tensor
  int k[kPerWave], v[kPerWave];
};

template <int D>
__device__ __forceinline__ FTileOff<D> ftile_offsets() {
  constexpr int RPL = FCfg<D>::kRowsPerLoad, CH = FCfg<D>::kChunks;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  const int rsub = l / CH, pc = l % CH;
  FTileOff<D> o;
#pragma unroll
  for (int q = 0; q < FTileOff<D>::kPerWave; ++q) {
    const int r = (wave * FTileOff<D>::kPerWave + q) * RPL + rsub;
    o.k[q] = (r * D + 8 * k_swz<D>(r, pc)) * 2;
    o.v[q] = (r * D + 8 * v_swz<D>(r, pc)) * 2;
  }
  return o;
}

template <int D>
__device__ __forceinline__ void ftile_issue(const uint16_t *base, int nvalid, char *buf,
                                            const int (&voff)[FTileOff<D>::kPerWave]) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const __amdgpu_buffer_rsrc_t rs =  // base and extent are uniform
      __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, nvalid * FCfg<D>::kRowBytes, kBufferRsrcWord3);
#pragma unroll
  for (int q = 0; q < FTileOff<D>::kPerWave; ++q)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)(buf + (wave * FTileOff<D>::kPerWave + q) * 1024), 16,
                                             voff[q], 0, 0, 0);
}

// Lazy softmax bound: the reference maximum is only raised when a lane's tile
// sum of exp2 terms exceeds 2^16 (or is not finite), so every P stays below
// 2^16 and the running sums stay far from overflow; the final division by l
// removes the common factor exactly.
constexpr float kLazyLimit = 65536.0f;

// s_waitcnt immediate (gfx9 encoding): at most n vector-memory operations
// outstanding and no LDS operation outstanding (expcnt left alone).
constexpr int waitcnt_vm_lgkm0(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

// Workgroup barrier for the K/V stages.  Each thread has already waited for
// its own direct-to-LDS loads of the stage about to be read (and for its LDS
// reads), so the barrier needs no memory fence; the "memory" clobber keeps
// the compiler from moving LDS accesses across it, and leaving out the fence
// keeps it from also waiting for the next stage's loads, which stay in flight.
__device__ __forceinline__ void stage_barrier() { asm volatile("s_barrier" ::: "memory"); }

template <int D>
__global__ __launch_bounds__(64 * kFWaves, 1) void k_attn_mfma(dkv_bank bank, const uint16_t *q, int nq,
                                                               KvSeg win, KvSeg sink,
                                                               uint16_t *out, float c, Geom g) {
  constexpr int KS = D / 16;   // K steps of S
  constexpr int DT = D / 32;   // dv tiles of O
  constexpr int RB = FCfg<D>::kRowBytes;
  constexpr int TB = FCfg<D>::kTileBytes;
  // direct-to-LDS loads per thread for one K + V tile
  constexpr int kTileLoads = 2 * (FCfg<D>::kLoadsPerTile / kFWaves);
  static_assert(FCfg<D>::kLoadsPerTile % kFWaves == 0, "tile loads must split evenly over the waves");
  // Workgroup L is dispatched to XCD L % 8.  Rank the workgroups XCD by XCD
  // (p = workgroups on lower XCDs + L / 8) and give rank p bank p / nqb, query
  // block p % nqb: the query blocks of a bank then run on one XCD and share
  // its L2 for the bank's keys and values.
  const int nqb = (nq + kFQ - 1) / kFQ;
  const int T = (int)gridDim.x, L = (int)blockIdx.x, xcd = L % 8;
  const int p = xcd * (T / 8) + min(xcd, T % 8) + L / 8;
  const int b = p / nqb, qblk = p % nqb;
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63, h = l >> 5, n = l & 31;
  const int M = clampi(bank.budget[b], 0, g.Mcap);
  const int m = clampi(bank.occupancy[b], 0, M);
  const int nw = win.n, ns = sink.n;
  const size_t rb = (size_t)b * g.Mcap, wb = (size_t)b * nw, sb = (size_t)b * ns;
  const uint16_t *wk = static_cast<const uint16_t *>(win.k), *wv = static_cast<const uint16_t *>(win.v);
  const uint16_t *sk = static_cast<const uint16_t *>(sink.k), *sv = static_cast<const uint16_t *>(sink.v);
  const uint16_t *bk = static_cast<const uint16_t *>(bank.k);
  const uint16_t *bv = static_cast<const uint16_t *>(bank.v);
  // One LDS array per stage (not one indexed array): with the stage known at
  // compile time the compiler can tell that reads of one stage never wait for
  // the direct-to-LDS loads still filling the others.
  __shared__ __attribute__((aligned(1024))) char k0[TB], k1[TB], k2[TB];
  __shared__ __attribute__((aligned(1024))) char v0[TB], v1[TB], v2[TB];

  const int qi = qblk * kFQ + wave * 32 + n;
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
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // Tiles never straddle the bank/window boundary: ceil(m/64) bank tiles, then
  // ceil(nw/64) window tiles, so every tile has one (scalar) base pointer.
  const int nt0 = (m + kFK - 1) / kFK;
  const int nt1 = nt0 + (nw + kFK - 1) / kFK;
  const int nt = nt1 + (ns + kFK - 1) / kFK;
  auto nvalid_of = [&](int t) {
    return t < nt0 ? min(kFK, m - t * kFK) : (t < nt1 ? min(kFK, nw - (t - nt0) * kFK) : min(kFK, ns - (t - nt1) * kFK));
  };
  const FTileOff<D> toff = ftile_offsets<D>();
  auto issue = [&](int t, char *kd, char *vd) {
    if (t >= nt) return;
    const int nv = nvalid_of(t);
    if (t < nt0) {
      ftile_issue<D>(bk + (rb + (size_t)t * kFK) * D, nv, kd, toff.k);
      ftile_issue<D>(bv + (rb + (size_t)t * kFK) * D, nv, vd, toff.v);
    } else if (t < nt1) {
      const size_t r0 = wb + (size_t)(t - nt0) * kFK;
      ftile_issue<D>(wk + r0 * D, nv, kd, toff.k);
      ftile_issue<D>(wv + r0 * D, nv, vd, toff.v);
    } else {
      const size_t r0 = sb + (size_t)(t - nt1) * kFK;
      ftile_issue<D>(sk + r0 * D, nv, kd, toff.k);
      ftile_issue<D>(sv + r0 * D, nv, vd, toff.v);
    }
  };
  // transposed V read: lane group gq = l / 16 (h = gq / 2), member cq = l % 16
  const int gq = l >> 4, cq = l & 15;

  // Tile t lives in stage t % 3.  Wait for its loads (the loads of tile t + 1
  // may stay in flight), then at the barrier every wave has finished tile
  // t - 1, so its stage receives tile t + 2.  Then S^T = K Q^T, softmax
  // update, O^T += V^T P^T.
  auto step = [&](int t, const char *kt, const char *vtile, char *kn, char *vn) {
    if (t + 1 < nt) __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(kTileLoads));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
    stage_barrier();
    issue(t + 2, kn, vn);
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
    // S block: LDS fragment reads run 6 MFMAs ahead of their use
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
    for (int i = 0; i < 2 * KS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i + 6 < 2 * KS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    const int nvalid = nvalid_of(t);
    if (nvalid < kFK) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (32 * sub + 8 * (i >> 2) + 4 * h + (i & 3) >= nvalid) sc[sub][i] = -INFINITY;
    }
    uint32_t pb[2][8];
    float psum = 0.0f;
    auto exps = [&](float moff) {
      float ps[2] = {0.0f, 0.0f};
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int i = 0; i < 16; i += 2) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[sub][i], c, moff));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[sub][i + 1], c, moff));
          pb[sub][i >> 1] = pack_bf16x2(p0, p1);
          // row sum of the bf16 weights actually multiplied into O
          ps[sub] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pb[sub][i >> 1]), ones, ps[sub], false);
        }
      psum = ps[0] + ps[1];
    };
    exps(-mrun * c);
    if (__any(!(psum <= kLazyLimit))) {
      float tmax = sc[0][0];
#pragma unroll
      for (int i = 1; i < 16; ++i) tmax = fmaxf(tmax, sc[0][i]);
#pragma unroll
      for (int i = 0; i < 16; ++i) tmax = fmaxf(tmax, sc[1][i]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      const float mnew = fmaxf(mrun, tmax);
      const float corr = __builtin_amdgcn_exp2f((mrun - mnew) * c);
      mrun = mnew;
      lrun *= corr;
#pragma unroll
      for (int t2 = 0; t2 < DT; ++t2)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[t2][i] *= corr;
      exps(-mrun * c);
    }
    lrun += psum;
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
    // P V block: the two transposed reads of an MFMA run 4 MFMAs ahead of it
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int i = 0; i < 4 * DT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i + 4 < 4 * DT) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
  };

  static_assert(kFStages == 3, "the loop below cycles through three stage buffers");
  issue(0, k0, v0);
  issue(1, k1, v1);
  for (int t = 0; t < nt; t += kFStages) {
    step(t, k0, v0, k2, v2);
    if (t + 1 < nt) step(t + 1, k1, v1, k0, v0);
    if (t + 2 < nt) step(t + 2, k2, v2, k1, v1);
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
hipError_t attn_impl(const dkv_bank &bank, const void *q, int nq, KvSeg win, KvSeg sink,
                     void *out, float scale, const Geom &g, hipStream_t s) {
  if (nq <= 0) return hipSuccess;
  const float scale_log2 = scale * 1.4426950408889634f;
  if constexpr (DT == DKV_BF16) {
    const long long nwg = (long long)((nq + kFQ - 1) / kFQ) * g.B;   // one-dimensional grid
    if (nwg > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nwg);
    k_attn_mfma<D><<<grid, 64 * kFWaves, 0, s>>>(bank, static_cast<const uint16_t *>(q), nq,
                                                 win, sink, static_cast<uint16_t *>(out), scale_log2, g);
  } else {
    dim3 grid((unsigned)((nq + kAThreads - 1) / kAThreads), (unsigned)g.B);
    k_attn_rowwise<D, DT><<<grid, kAThreads, 0, s>>>(bank, q, nq, win, sink, out, scale_log2, g);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const dkv_bank &bank, const void *q, int nq, KvSeg win, KvSeg sink, void *out,
                            float scale, const Geom &g, hipStream_t s) {
  if (g.d == 128 && g.dtype == DKV_BF16) return attn_impl<128, DKV_BF16>(bank, q, nq, win, sink, out, scale, g, s);
  if (g.d == 128 && g.dtype == DKV_F32) return attn_impl<128, DKV_F32>(bank, q, nq, win, sink, out, scale, g, s);
  if (g.d == 64 && g.dtype == DKV_BF16) return attn_impl<64, DKV_BF16>(bank, q, nq, win, sink, out, scale, g, s);
  return attn_impl<64, DKV_F32>(bank, q, nq, win, sink, out, scale, g, s);
}

}  // namespace dkv
