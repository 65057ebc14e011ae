/*
 * densitykv.h -- C ABI of the DensityKV hot path on MI355X (gfx950).
 *
 * DensityKV keeps, for every (layer, head), a bank of at most M exact post-RoPE
 * key/value pairs (Sec. 3.4, Eq. 4).  Once per finalized generation block the
 * bank is updated from the block's N candidates (Sec. 3.4, Eqs. 5-12; Supp. C,
 * Algorithm 1), and the next block's queries attend over the retained bank
 * plus the local window with the backbone's native attention (Sec. 1, Fig. 1;
 * Sec. 3.2 logit).  This header exposes that path:
 *
 *   densitykv_score           Soft-Riesz candidate scores (Eq. 6) and, on
 *                             request, every bank state's density (Eq. 3);
 *   densitykv_update_bank     the full update of Algorithm 1 for all banks;
 *   densitykv_bank_attention  softmax(q k^T * scale) v over [bank; window];
 *   densitykv_bank_attention_sink  the same over [bank; window; sink].
 *
 * Conventions shared by every entry point
 *   - Every pointer inside the structs and every array argument is DEVICE
 *     memory owned by the caller.  The library never allocates, never frees
 *     and keeps no pointer after a call returns.
 *   - Every call only enqueues work on `stream` (a hipStream_t; NULL = the
 *     null stream) and returns without synchronising.  Outputs are valid once
 *     the stream has reached them.
 *   - Return value: DKV_OK or a negative dkv_status.  Arguments are checked on
 *     the host before anything is enqueued; on an error nothing is enqueued.
 *   - Row-major layouts; "[B, Mcap, d]" means bank b's slot s starts at
 *     element ((b * Mcap) + s) * d.  Keys and values share one dtype and d_k = d_v.
 *
 * Arithmetic (so that results are bit-reproducible against a plain CPU
 * evaluation of the paper's definitions):
 *   - keys are expected on the grid n/64, |n| <= 127 (exact in bf16 and fp32);
 *     every key-key Gram is then exact in any summation order.  Keys off the
 *     grid are accepted; decisions then carry fp32 Gram rounding;
 *   - the pair weight w = (1 + d2 / sigma^2)^-p (Eq. 2, eps = 1) is computed
 *     in IEEE binary32 with round-to-nearest-even at every step, and a
 *     correctly rounded reciprocal;
 *   - densities, baselines and scores are int64 sums of Q23 fixed-point terms
 *     (weight 1.0 == 2^23), so no decision depends on summation order.
 */
#ifndef DENSITYKV_H
#define DENSITYKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DKV_OK = 0,
  DKV_ERR_INVALID = -1,     /* NULL pointer, bad enum, unknown policy flags     */
  DKV_ERR_SHAPE = -2,       /* sizes out of range or inconsistent               */
  DKV_ERR_UNSUPPORTED = -3, /* head_dim, p or sigma^2 not supported             */
  DKV_ERR_WORKSPACE = -4,   /* workspace NULL or smaller than required          */
  DKV_ERR_RANGE = -5,       /* fixed-point range would overflow                 */
  DKV_ERR_HIP = -6,         /* a HIP launch reported an error                   */
  DKV_ERR_SCRATCH = -7      /* needs more than DKV_NOALLOC_SCRATCH_BYTES        */
} dkv_status;

typedef enum { DKV_BF16 = 0, DKV_F32 = 1 } dkv_dtype;

/* Limits checked on the host. */
#define DKV_MAX_CANDIDATES 8191   /* N per block (source index packs into 13 bits) */
#define DKV_MAX_CAPACITY 32767    /* Mcap (slot index packs into 15 bits)          */
#define DKV_MAX_BLOCK_ID 16777215 /* provenance block id < 2^24                    */

/*
 * Per-(layer, head) banks, B = num_banks of them (Sec. 3.4, Eq. 4).  Bank b
 * belongs to group b / group_size; the banks of one group (the heads of one
 * layer, group_size = H) admit the same number of candidates per update
 * (Eq. 11); group_size = 1 gives the independent per-head variant (Supp. E,
 * "Cross-head synchronization").  Only slots [0, occupancy[b]) are live.
 *
 *   k, v       [B, Mcap, d] dtype      exact post-RoPE keys and their values
 *   knorm      [B, Mcap]    float      |k|^2 of each live slot (maintained)
 *   rho        [B, Mcap]    int64      current density Phi over the bank, Q23
 *   base       [B, Mcap]    int64      frozen insertion baseline (Eq. 5), Q23
 *   prov       [B, Mcap]    int64      (block_id << 32) | source index
 *   occupancy  [B]          int32      m_b, read and rewritten on the device
 *   budget     [B]          int32      M_b; clamped on the device to [0, Mcap]
 * A fresh bank is all zeros with occupancy 0.  occupancy is clamped on the
 * device to [0, M_b].  Within a group the prefix length r never exceeds any
 * member's budget; with equal budgets this is exactly Eq. 11.
 */
typedef struct {
  int32_t num_banks; /* B >= 1, with B * max(capacity, DKV_MAX_CANDIDATES) < 2^31 */
  int32_t group_size;
  int32_t head_dim;  /* 64 or 128 */
  int32_t capacity;  /* Mcap, row stride of every per-slot array, 1..DKV_MAX_CAPACITY */
  int32_t dtype;     /* dkv_dtype */
  void *k;
  void *v;
  float *knorm;
  int64_t *rho;
  int64_t *base;
  int64_t *prov;
  int32_t *occupancy;
  const int32_t *budget;
} dkv_bank;

/* One finalized block of N candidates per bank, in source order (Sec. 3.4:
 * the block leaving the local window).  k, v: [B, n, d] in the bank dtype. */
typedef struct {
  int32_t n;        /* 0..DKV_MAX_CANDIDATES */
  int32_t block_id; /* 0..DKV_MAX_BLOCK_ID, recorded in the provenance */
  const void *k;
  const void *v;
} dkv_segment;

/* Method parameters (Sec. 3.3-3.4; defaults of Sec. 4.1: eps = 1 fixed,
 * p = 2, sigma = 8 -> sigma^2 = 2^6, tau = 2, delta = 1e-6 -> delta_q = 8). */
typedef struct {
  int32_t sigma2_log2;  /* sigma^2 = 2^sigma2_log2, -8..16 */
  int32_t p;            /* 1, 2 or 4 */
  int32_t tau_num;      /* tau = tau_num / 2^tau_log2_den, tau > 1, tau_num <= 2^16 */
  int32_t tau_log2_den; /* 0..8 */
  int64_t delta_q;      /* baseline floor in Q23 units, 1..2^40 */
  uint32_t flags;       /* 0 (the paper's policy) or DKV_POLICY_* bits below */
} dkv_params;

/* Policy ablations of Table 1(b), defined in the supplementary ablation details
 * (Supp. E: "Candidate ordering", "Density baseline", "Eviction rule").  They
 * change only the prefix order, the baseline update or the eviction fill; the
 * Gram stages, the prefix feasibility test (Eqs. 8-11) and the maintenance are
 * the same.  DENSEST_ONLY and SOURCE_FILL are exclusive; any other bit is
 * rejected with DKV_ERR_INVALID.  (The independent per-head variant is
 * group_size = 1.)  SEQUENTIAL (below) replaces the prefix test itself.
 *   SOURCE_ORDER  the tested prefixes follow the candidates' source order
 *                 instead of the score order (scores are still computed and
 *                 reported in score_q)
 *   REFRESH_BASE  after the update every retained state's baseline is
 *                 recomputed from its maintained density: b = max(rho, delta)
 *   DENSEST_ONLY  no mandatory set: the e_{r*} states of largest rho~(r*) are
 *                 released (ties: smaller provenance, then lower slot); a
 *                 violator outside them stays in the bank
 *   SOURCE_FILL   all violators, then the non-violators in admission order
 *                 (ascending provenance, then slot) until e_{r*} are released
 *   KV_DESCRIPTOR the retention geometry uses the concatenated [k; v] row
 *                 (2 d elements; Supp. E "Retention geometry", the post-RoPE
 *                 [K;V] rows of Table 1(b)) for every density, score and
 *                 crossing; attention is unchanged.  bf16 banks only
 *                 (DKV_ERR_UNSUPPORTED otherwise); the values must then lie on
 *                 the key grid for exact decisions, the segment's v is
 *                 required (DKV_ERR_INVALID), and knorm holds |k|^2 + |v|^2, so
 *                 a bank must be updated and scored with one geometry. */
#define DKV_POLICY_SOURCE_ORDER 0x1u
#define DKV_POLICY_REFRESH_BASE 0x2u
#define DKV_POLICY_DENSEST_ONLY 0x4u
#define DKV_POLICY_SOURCE_FILL 0x8u
#define DKV_POLICY_KV_DESCRIPTOR 0x10u
/* Within-block sequential competition (Supp. E, "Within-block competition";
 * Supp. C, "Insertion hysteresis"): candidates are admitted one at a time, each
 * tested against the bank as the previous admissions of the same block left
 * it.  The candidates keep the order above, fixed at the start of the
 * block, and are offered one at a time: step j tests the j-th candidate x of
 * every bank of the group as a one-candidate prefix against that bank as it is
 * at that step (earlier admissions included, with exactly maintained
 * densities and baselines frozen when they entered).  Violators are the states
 * with 2^k (rho_i + W_ix) >= T b_i and e = max(0, m + 1 - M) <= 1; the step is
 * taken iff every bank of the group has at most e violators.  Then each bank
 * releases its violator, or with none and e = 1 its state of largest
 * rho_i + W_ix (ties: smaller provenance, then lower slot); survivors get
 * rho_i += W_ix - W_i,released; x gets rho = sum of W_xi over the survivors and
 * b = max(rho, delta), in the released slot or the next free one.  A rejected
 * step drops its candidates.  A bank that is empty at the start of the block
 * takes the empty-bank rule and stays out of the shared test.  Combines with
 * SOURCE_ORDER and REFRESH_BASE only (DKV_ERR_INVALID otherwise); bf16 banks
 * only (DKV_ERR_UNSUPPORTED); group_size <= 256 (DKV_ERR_SHAPE).
 * Workspace: 12 bytes per slot and 8 KiB per group, plus an area for the
 * pairwise weights of [bank; candidates] of whole groups,
 * group_size * (capacity + n)^2 * 4 bytes per group.  The groups are updated
 * in batches of as many as that area holds: densitykv_update_bank takes the
 * batch from the workspace_bytes it is given (every byte beyond the fixed part
 * goes to the area; DKV_ERR_WORKSPACE when not even one group fits), and
 * densitykv_workspace_size_policy asks for the groups that fit in
 * DKV_SEQ_WEIGHT_BYTES (at least one, at most all).  A larger workspace walks
 * more groups at once.
 * Outputs: r_star = steps taken, n_admitted / admitted = this block's
 * candidates in the final bank, n_evicted / evicted = pre-update slots whose
 * state left; first_cross and rho_tilde are not written.  The steps are
 * inherently sequential: the workgroups that hold a group's banks exchange
 * one record per step through the workspace (when all of them fit on the
 * device at once; otherwise one workgroup walks the group).  r_star = -1
 * reports a walk whose wait for those records exceeded its bound, leaving
 * the group's banks undefined; with the launch guarantees in place this does
 * not occur.  The call itself cannot report it (the walk runs after the call
 * returns): a caller that must know passes r_star and reads it after the
 * stream has completed.  Which walk runs is decided before anything is
 * enqueued, and every write to a bank comes after the walk's launch. */
#define DKV_POLICY_SEQUENTIAL 0x20u
/* Pairwise-weight bytes that densitykv_workspace_size_policy sizes the
 * sequential competition's batches for (32 GiB). */
#define DKV_SEQ_WEIGHT_BYTES ((size_t)32 << 30)

/* Optional outputs of densitykv_update_bank (any pointer may be NULL).
 *   r_star       [G]        admitted prefix length of each group (Eq. 11)
 *   n_admitted   [B]        = r_star of the bank's group
 *   n_evicted    [B]        |R| of each bank
 *   admitted     [B, N]     admitted source indices, ascending, -1 padded
 *   evicted      [B, Mcap]  evicted pre-update slots, ascending, -1 padded
 *   order        [B, N]     candidate order pi (source indices; identity for an empty bank)
 *   score_q      [B, N]     fixed-point candidate score S_x (0 for an empty bank)
 *   first_cross  [B, Mcap]  per pre-update slot: smallest prefix length r at which
 *                           the state violates the growth bound, R+1 if none
 *                           within r <= R (R = min(N, budgets of the group))
 *   rho_tilde    [B, Mcap]  per pre-update slot: rho + sum of its weights to the
 *                           admitted prefix (projected density at r*, Q23)
 * Without first_cross the crossing search may end after the first 256 ordered
 * candidates for a group that some bank's crossings there already rule out of
 * every longer prefix (Eqs. 9-11); every other output is the same either way. */
typedef struct {
  int32_t *r_star;
  int32_t *n_admitted;
  int32_t *n_evicted;
  int32_t *admitted;
  int32_t *evicted;
  int32_t *order;
  int64_t *score_q;
  int32_t *first_cross;
  int64_t *rho_tilde;
} dkv_update_out;

/* Bytes of device workspace densitykv_score / densitykv_update_bank need for
 * this bank geometry and n_cand candidates per bank.  Host-only; enqueues nothing. */
int densitykv_workspace_size(const dkv_bank *bank, int32_t n_cand, size_t *bytes);

/* The same for the given dkv_params.flags: larger with DKV_POLICY_SEQUENTIAL
 * (the fixed part plus the pairwise weights of as many whole groups as fit in
 * DKV_SEQ_WEIGHT_BYTES, at least one), equal to densitykv_workspace_size
 * otherwise.  Host-only. */
int densitykv_workspace_size_policy(const dkv_bank *bank, int32_t n_cand, uint32_t flags, size_t *bytes);

/*
 * Candidate scores against the current banks (Eq. 6; Supp. C), without
 * changing any bank.
 *   cand_score_q   [B, N] int64  S_x: fixed-point sum over the bank of
 *                                w(k_i, k_x) * (1/b_i) * 2^(23-E_b), E_b the
 *                                binary exponent of max_i 1/b_i of bank b;
 *                                S_x = 2^(23-E_b) * m_b * s_h(x) up to per-term
 *                                rounding.  Ties are broken by source order in
 *                                the update.  0 for an empty bank.  May be NULL.
 *   cand_score_f32 [B, N] float  s_h(x) = S_x * 2^(E_b-23) / m_b (0 for an empty
 *                                bank).  May be NULL.
 *   bank_density_q [B, Mcap] int64  Phi over the bank (Eq. 3) of every live slot,
 *                                recomputed from scratch (O(m^2) pairs); slots
 *                                >= m_b are left untouched.  May be NULL.
 */
int densitykv_score(const dkv_bank *bank, const dkv_segment *seg, const dkv_params *prm,
                    int64_t *cand_score_q, float *cand_score_f32, int64_t *bank_density_q,
                    void *workspace, size_t workspace_bytes, void *stream);

/*
 * One DensityKV update of every bank from one block (Supp. C, Algorithm 1):
 * order candidates by score (empty bank: source order), find the largest
 * prefix length feasible for every bank of the group (Eqs. 8-11), evict all
 * violators and then the densest states until e_{r*} are released (Sec. 3.4
 * step 3; fill ties: earlier provenance, then lower slot), commit (Eq. 12)
 * and maintain every density exactly (Supp. C).  Commit layout: survivors keep
 * their slots; admitted candidates in ascending source index fill the evicted
 * slots in ascending order, then are appended; if more states were evicted
 * than admitted, the states at or beyond the new occupancy move into the
 * remaining holes (ascending).  The bank is modified in place; `out` may be
 * NULL.  r* never leaves the device.
 */
int densitykv_update_bank(dkv_bank *bank, const dkv_segment *seg, const dkv_params *prm,
                          dkv_update_out *out, void *workspace, size_t workspace_bytes,
                          void *stream);

/*
 * densitykv_update_bank for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same update, with its workspace taken from a static device
 * buffer of DKV_NOALLOC_SCRATCH_BYTES that the library holds on every device
 * it runs on until the process ends.  The call itself allocates and frees
 * nothing.  The caller still passes the bank, the segment and the outputs.
 *   - Uses the scratch of the current device; `stream` must belong to it.
 *   - Returns DKV_ERR_SCRATCH, before enqueueing anything, when
 *     densitykv_workspace_size_policy(bank, seg->n, prm->flags) exceeds
 *     DKV_NOALLOC_SCRATCH_BYTES (e.g. 12 banks of 4,680 slots with 4,680
 *     candidates, d = 128, fit; 360 such banks do not).  Other errors as
 *     densitykv_update_bank.
 *   - Every call on one device shares that device's scratch; the update
 *     initialises every part of it that it reads, so the contents a previous
 *     call left do not matter.  Calls that overlap in time on one device
 *     (different streams, or several host threads) race on it: serialise them.
 */
#define DKV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int densitykv_update_bank_noalloc(dkv_bank *bank, const dkv_segment *seg, const dkv_params *prm,
                                  dkv_update_out *out, void *stream);

/*
 * Native attention of n_query queries per bank over the bank's live slots
 * followed by n_window window tokens (Sec. 1, Fig. 1: native attention reads
 * the retained bank with the local window; Sec. 3.2: logit q^T k / sqrt(d_k)):
 *   out = softmax(q K^T * softmax_scale) V,  K = [bank k[0:m_b]; win_k],  V likewise.
 *   q, out         [B, n_query, d]   bank dtype (bf16: fp32 softmax and accumulation)
 *   win_k, win_v   [B, n_window, d]  bank dtype; may be NULL when n_window = 0
 * A bank with m_b + n_window = 0 yields zeros.  No mask, sink or RoPE is applied.
 */
int densitykv_bank_attention(const dkv_bank *bank, const void *q, int32_t n_query,
                             const void *win_k, const void *win_v, int32_t n_window,
                             void *out, float softmax_scale, void *stream);

/*
 * The same attention in the paper's deployment context (Supp. D, memory
 * budget and temporal alignment): a first-frame sink, the local window and the
 * retained bank read together, out = softmax(q K^T * scale) V with
 * K = [bank k[0:m_b]; window k; sink k].  Arguments as densitykv_bank_attention,
 * plus
 *   sink_k, sink_v [B, n_sink, d]  bank dtype; may be NULL when n_sink = 0
 * Keys are used as given (already post-RoPE, memory keys with the temporal
 * coordinate set as the backbone does); no mask is applied.  Same errors as
 * densitykv_bank_attention, and DKV_ERR_INVALID for a NULL sink with
 * n_sink > 0.  densitykv_bank_attention is this call with n_sink = 0.
 */
int densitykv_bank_attention_sink(const dkv_bank *bank, const void *q, int32_t n_query,
                                  const void *sink_k, const void *sink_v, int32_t n_sink,
                                  const void *win_k, const void *win_v, int32_t n_window,
                                  void *out, float softmax_scale, void *stream);

/*
 * The per-pair contract on its own: w_q23[i] = RNE(w(d2[i]) * 2^23) with
 * w = (1 + d2/sigma^2)^-p in binary32 (Eq. 2, eps = 1).  d2 [n] float,
 * w_q23 [n] int32, both device memory.  Used to check the kernels' weight
 * arithmetic exhaustively over every squared distance the key grid can produce.
 */
int densitykv_pair_weight_q23(const float *d2, int64_t n, const dkv_params *prm,
                              int32_t *w_q23, void *stream);

/* Static text for a dkv_status value. */
const char *densitykv_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* DENSITYKV_H */
