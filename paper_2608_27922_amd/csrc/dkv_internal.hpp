// Internal declarations shared by the DensityKV HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/densitykv.h"

namespace dkv {

constexpr uint32_t kQ23 = 1u << 23;          // weight 1.0 in fixed point
constexpr uint32_t kMagic = 0x4B000000u;     // bit pattern of 2^23 as binary32
constexpr int kCkStride = 64;                // prefix checkpoint spacing (candidates)
constexpr int kSortMax = 8192;               // padded sort size (N <= 8191)

// ---------------------------------------------------------------------------
// Workspace: one carve of the caller's buffer, every array 256-byte aligned.
// ---------------------------------------------------------------------------
struct Workspace {
  int32_t *m;          // [B] occupancy on entry (clamped)
  int32_t *M;          // [B] budget (clamped to [0, Mcap])
  int32_t *R;          // [B] largest tested prefix of the bank's group
  int32_t *E;          // [B] score exponent
  int32_t *e;          // [B] e_{r*}
  int32_t *r_star;     // [G]
  int32_t *n_ev;       // [B]
  int32_t *m_new;      // [B]
  float *cnorm;        // [B, N]   |k_x|^2 of candidates
  float *bs;           // [B, Mcap] score scale of each bank state
  int64_t *acol;       // [B, N]   S_x
  int32_t *order;      // [B, N]   pi
  int32_t *rank;       // [B, N]   position of x in pi
  int32_t *first;      // [B, Mcap] first crossing prefix length
  uint32_t *ck;        // [B, Mcap, nck] sums over each kCkStride-candidate chunk of the order
  int64_t *rho_t;      // [B, Mcap] rho + P(r*)
  int32_t *dest;       // [B, Mcap] final slot of each pre-update slot, -1 if evicted
  int32_t *ev_list;    // [B, Mcap] evicted slots ascending
  int32_t *surv_list;  // [B, Mcap] surviving slots ascending
  int32_t *adm_list;   // [B, N]   admitted source indices ascending
  int32_t *adm_dest;   // [B, N]   final slot of each admitted candidate
  int64_t *sub;        // [B, Mcap] sum of weights to the evicted states (survivors)
  int64_t *sub_adm;    // [B, N]   admitted: sum of weights to the survivors
  int64_t *mut_adm;    // [B, N]   admitted: sum of weights to the other admitted
  int32_t *hole_list;  // [B, Mcap] holes closed by moving states (states violating before the update)
  uint16_t *sk;        // [B, N, d] bf16 candidate keys in score order
  float *snorm;        // [B, N]   their norms
  uint4 *baug;         // [B, Mcap] column aug step of each bank state (column_aug)
  uint4 *caug;         // [B, N]   of each candidate, source order
  uint4 *saug;         // [B, N]   of each candidate, score order
  int32_t *maint_off;  // [B + 1] first maintenance work item of each bank; [B] = total
  int32_t *crossed;    // [B] states whose first crossing lies in the first part of the crossing search
  int32_t *more;       // [G] 1 where the group's crossing search needs the prefixes past its first part
  uint32_t *feas;      // [B, nfw] bit r: prefix length r feasible for this bank
  int nfw;             // words per bank of feas
  uint64_t *skeys;     // [B, npad] sort keys, sorted within 512-key chunks
  int npad;            // N rounded up to 512
  int nck;
  // sequential competition only (null otherwise)
  uint32_t *gram;      // [Bw, L, L] W between the items [slots 0..Mcap); candidates 0..N)], L = Mcap + N,
                       // for the Bw banks seq_b0 .. seq_b0 + Bw - 1 of the batch being walked
  int32_t *grow;       // [B, Mcap] item of the state in each slot (slot s, or Mcap + candidate)
  int64_t *lim;        // [B, Mcap] ceil(T b / 2^k): the state violates when rho + W reaches it
  uint64_t *seq_rec;   // [G, 2, kSeqMaxMembers, 8] per-step records of the workgroups of a group
  int gram_ld;         // L
  int seq_b0;          // first bank of the batch whose weights gram holds
  int seq_groups;      // groups per batch (whole groups whose weights fit in gram)
};

// seq_groups: groups whose pairwise weights the sequential competition's area
// holds (0 for none); the area comes last, after every fixed-size array.
size_t workspace_layout(int B, int G, int Mcap, int N, int d, Workspace *ws, char *base, bool seq = false,
                        int seq_groups = 0);
// Bytes of the pairwise weights of one group in the sequential competition.
inline size_t seq_group_weight_bytes(int gs, int Mcap, int N) {
  const size_t L = (size_t)Mcap + (size_t)(N > 0 ? N : 0);
  return (size_t)gs * L * L * 4;
}
constexpr int kSeqMaxGroup = 256;  // banks per group in the sequential competition
constexpr int kSeqMaxMembers = 64;  // workgroups per group in the multi-workgroup walk

// Geometry and parameters passed by value to every kernel.
struct Geom {
  int B, G, gs, d, Mcap, N, dtype;
};
struct Prm {
  float inv_sigma2;  // 2^-sigma2_log2 (exact)
  int p;
  int tau_num, tau_shift;
  int64_t delta_q;
  int block_id;
  uint32_t flags;  // DKV_POLICY_* bits
};

// Launchers (host functions defined in the .hip sources; return hipError_t).
hipError_t launch_update(const dkv_bank &bank, const dkv_segment &seg, const Geom &g,
                         const Prm &p, const dkv_update_out *out, const Workspace &ws,
                         hipStream_t s);
hipError_t launch_score(const dkv_bank &bank, const dkv_segment &seg, const Geom &g,
                        const Prm &p, int64_t *score_q, float *score_f32, int64_t *density,
                        const Workspace &ws, hipStream_t s);
// One extra key/value segment of the attention context: [B, n, d] device arrays.
struct KvSeg {
  const void *k;
  const void *v;
  int n;
};
hipError_t launch_attention(const dkv_bank &bank, const void *q, int nq, KvSeg win, KvSeg sink,
                            void *out, float scale, const Geom &g, hipStream_t s);
void launch_gram_mfma(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                      const dkv_update_out &out, const Workspace &ws, hipStream_t s, int stage);
void launch_score_mfma(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                       int64_t *score_q, float *score_f, int64_t *density, const Workspace &ws, hipStream_t s);
hipError_t launch_pair_weight(const float *d2, int64_t n, const Prm &p, int32_t *w,
                              hipStream_t s);
// Within-block sequential competition after the order is known (bf16 banks).
hipError_t launch_sequential(const dkv_bank &bank, const dkv_segment &seg, const Geom &g, const Prm &p,
                             const dkv_update_out &out, const Workspace &ws, hipStream_t s);

#if defined(__HIPCC__)
// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}
// Two floats -> packed bf16 pair (low half first), round to nearest even
// (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {  // RNE, finite inputs
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
template <int DT>
__device__ __forceinline__ float load_elem(const void *p, size_t i) {
  if constexpr (DT == DKV_BF16) {
    return bf16_bits_to_f32(static_cast<const uint16_t *>(p)[i]);
  } else {
    return static_cast<const float *>(p)[i];
  }
}

// Correctly rounded binary32 reciprocal for normal inputs with normal results:
// one Newton-Raphson step y + y (1 - x y) on the hardware estimate y, with the
// residual 1 - x y computed exactly by a fused multiply-add (Markstein's
// correction scheme, IBM J. Res. Dev. 34(1), 1990).  Checked against the IEEE
// division for every significand.
__device__ __forceinline__ float rcp_rn(float x) {
  const float y = __builtin_amdgcn_rcpf(x);
  const float e = __builtin_fmaf(-x, y, 1.0f);
  return __builtin_fmaf(e, y, y);
}
// A weight is at most eps^-p = 1 (t = 1 + d2 / sigma^2 >= 1).  On the key grid
// t >= 1 holds exactly; off the grid the fp32 Gram can round d2 below 0 for
// near-duplicates, so the weight is clamped to [0, 1].  The clamp is the output
// modifier of the last FMA (no extra instruction) and keeps every fixed-point
// weight within 2^23, as the Q23 rounding and the packed record fields need.
__device__ __forceinline__ float clamp_weight(float w) { return __builtin_amdgcn_fmed3f(w, 0.0f, 1.0f); }

// Soft-Riesz weight (eps = 1): w = 1 / (1 + d2 / sigma^2)^p, each step one
// binary32 operation rounded to nearest even with a correctly rounded
// reciprocal.  d2 * inv_sigma2 is exact (power of two).
__device__ __forceinline__ float pair_weight(float d2, float inv_sigma2, int p) {
  float t = 1.0f + d2 * inv_sigma2;
  float tp = t;
  if (p >= 2) tp = t * t;
  if (p == 4) tp = tp * tp;
  return clamp_weight(rcp_rn(tp));
}
// Score scale of a bank state (Eq. 6): fp32(2^23 / b) by one fp64 division
// rounded to fp32, times 2^(23 - E) with E the binary exponent of the bank's
// largest such value (so the scale is at most 2^23).  Baselines below 1 read as 1.
__device__ __forceinline__ float score_scale(int64_t base, int E) {
  const int64_t bi = base < 1 ? 1 : base;
  return ldexpf((float)(8388608.0 / (double)bi), 23 - E);
}
// RNE(w * scale) for w * scale in [0, 2^23]: fma(w, scale, 2^23) lands in
// [2^23, 2^24] where one ulp is 1, so its bit pattern minus that of 2^23 is
// the rounded integer.
__device__ __forceinline__ uint32_t q23_round(float w, float scale) {
  return __float_as_uint(__builtin_fmaf(w, scale, 8388608.0f)) - kMagic;
}
// Column item's extra K step of the MFMA Gram (bf16 x 8): its norm / sigma^2
// split exactly into three bf16 pieces, then four ones (the row item's norm
// pieces and the folded 1 of t = 1 + u), then 0.
__device__ __forceinline__ uint4 column_aug(float norm, float inv_s2) {
  const float x = norm * inv_s2;
  const uint16_t h = f32_to_bf16_bits(x);
  const float r = x - bf16_bits_to_f32(h);
  const uint16_t m = f32_to_bf16_bits(r);
  const uint16_t l = f32_to_bf16_bits(r - bf16_bits_to_f32(m));
  constexpr uint32_t one = 0x3F80u;
  return uint4{(uint32_t)h | ((uint32_t)m << 16), (uint32_t)l | (one << 16), one | (one << 16), one};
}
#endif

}  // namespace dkv
