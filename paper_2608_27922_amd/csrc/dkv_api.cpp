// C ABI of the DensityKV hot path: argument checks, workspace carving and the
// enqueueing of the kernel sequences (see include/densitykv.h for the contract).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>

#include "dkv_internal.hpp"

namespace dkv {

static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t workspace_layout(int B, int G, int Mcap, int N, int d, Workspace *ws, char *base, bool seq,
                        int seq_groups) {
  size_t off = 0;
  const size_t Bz = (size_t)B, Mz = (size_t)Mcap, Nz = (size_t)(N > 0 ? N : 1);
  // chunk sums per row, padded to a multiple of 4 so that rows are 16-byte aligned
  const int nck = ((N + kCkStride - 1) / kCkStride + 3) / 4 * 4;
  auto take = [&](size_t bytes) -> char * {
    char *p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  };
  Workspace w{};
  w.m = (int32_t *)take(Bz * 4);
  w.M = (int32_t *)take(Bz * 4);
  w.R = (int32_t *)take(Bz * 4);
  w.E = (int32_t *)take(Bz * 4);
  w.e = (int32_t *)take(Bz * 4);
  w.r_star = (int32_t *)take((size_t)G * 4);
  w.n_ev = (int32_t *)take(Bz * 4);
  w.m_new = (int32_t *)take(Bz * 4);
  w.cnorm = (float *)take(Bz * Nz * 4);
  w.bs = (float *)take(Bz * Mz * 4);
  w.acol = (int64_t *)take(Bz * Nz * 8);
  w.order = (int32_t *)take(Bz * Nz * 4);
  w.rank = (int32_t *)take(Bz * Nz * 4);
  w.first = (int32_t *)take(Bz * Mz * 4);
  w.ck = (uint32_t *)take(Bz * Mz * (size_t)(nck > 0 ? nck : 4) * 4);
  w.rho_t = (int64_t *)take(Bz * Mz * 8);
  w.dest = (int32_t *)take(Bz * Mz * 4);
  w.ev_list = (int32_t *)take(Bz * Mz * 4);
  w.surv_list = (int32_t *)take(Bz * Mz * 4);
  w.adm_list = (int32_t *)take(Bz * Nz * 4);
  w.adm_dest = (int32_t *)take(Bz * Nz * 4);
  w.sub = (int64_t *)take(Bz * Mz * 8);
  w.sub_adm = (int64_t *)take(Bz * Nz * 8);
  w.mut_adm = (int64_t *)take(Bz * Nz * 8);
  w.hole_list = (int32_t *)take(Bz * Mz * 4);
  w.sk = (uint16_t *)take(Bz * Nz * (size_t)d * 4);  // ordered descriptors: up to [k; v], 2 d bf16
  w.snorm = (float *)take(Bz * Nz * 4);
  w.baug = (uint4 *)take(Bz * Mz * 16);
  w.caug = (uint4 *)take(Bz * Nz * 16);
  w.saug = (uint4 *)take(Bz * Nz * 16);
  w.maint_off = (int32_t *)take((Bz + 1) * 4);
  w.crossed = (int32_t *)take(Bz * 4);
  w.more = (int32_t *)take((size_t)G * 4);
  const int nfw = ((N > 0 ? N : 0) + 1 + 31) / 32;
  w.feas = (uint32_t *)take(Bz * (size_t)nfw * 4);
  w.nfw = nfw;
  const int npad = ((N > 0 ? N : 1) + 511) / 512 * 512;
  w.skeys = (uint64_t *)take(Bz * (size_t)npad * 8);
  w.npad = npad;
  w.nck = nck > 0 ? nck : 4;
  if (seq) {
    const size_t L = (size_t)Mcap + (size_t)(N > 0 ? N : 0);
    w.grow = (int32_t *)take(Bz * Mz * 4);
    w.lim = (int64_t *)take(Bz * Mz * 8);
    w.seq_rec = (uint64_t *)take((size_t)G * 2 * kSeqMaxMembers * 8 * 8);
    w.gram_ld = (int)L;
    w.seq_b0 = 0;
    w.seq_groups = seq_groups;
    // last: the pairwise weights of seq_groups whole groups
    w.gram = (uint32_t *)take((size_t)seq_groups * seq_group_weight_bytes(B / G, Mcap, N));
  }
  if (ws) *ws = w;
  return off;
}

}  // namespace dkv

using namespace dkv;

namespace {

int check_bank(const dkv_bank *bk) {
  if (!bk) return DKV_ERR_INVALID;
  if (bk->dtype != DKV_BF16 && bk->dtype != DKV_F32) return DKV_ERR_INVALID;
  if (bk->head_dim != 64 && bk->head_dim != 128) return DKV_ERR_UNSUPPORTED;
  if (bk->num_banks < 1 || bk->group_size < 1 || bk->num_banks % bk->group_size != 0) return DKV_ERR_SHAPE;
  if (bk->capacity < 1 || bk->capacity > DKV_MAX_CAPACITY) return DKV_ERR_SHAPE;
  // bank rows and candidate rows are indexed with 32-bit integers in the kernels
  const int64_t rows = (int64_t)bk->num_banks * (bk->capacity > DKV_MAX_CANDIDATES ? bk->capacity : DKV_MAX_CANDIDATES);
  if (rows >= (int64_t(1) << 31)) return DKV_ERR_SHAPE;
  if (!bk->k || !bk->v || !bk->knorm || !bk->rho || !bk->base || !bk->prov || !bk->occupancy || !bk->budget)
    return DKV_ERR_INVALID;
  return DKV_OK;
}

int check_segment(const dkv_segment *sg) {
  if (!sg) return DKV_ERR_INVALID;
  if (sg->n < 0 || sg->n > DKV_MAX_CANDIDATES) return DKV_ERR_SHAPE;
  if (sg->block_id < 0 || sg->block_id > DKV_MAX_BLOCK_ID) return DKV_ERR_RANGE;
  if (sg->n > 0 && (!sg->k || !sg->v)) return DKV_ERR_INVALID;
  return DKV_OK;
}

int check_params(const dkv_params *p, Prm *out, int block_id) {
  if (!p) return DKV_ERR_INVALID;
  const uint32_t known = DKV_POLICY_SOURCE_ORDER | DKV_POLICY_REFRESH_BASE | DKV_POLICY_DENSEST_ONLY |
                         DKV_POLICY_SOURCE_FILL | DKV_POLICY_KV_DESCRIPTOR | DKV_POLICY_SEQUENTIAL;
  if (p->flags & ~known) return DKV_ERR_INVALID;
  if ((p->flags & DKV_POLICY_DENSEST_ONLY) && (p->flags & DKV_POLICY_SOURCE_FILL)) return DKV_ERR_INVALID;
  if ((p->flags & DKV_POLICY_SEQUENTIAL) &&
      (p->flags & (DKV_POLICY_DENSEST_ONLY | DKV_POLICY_SOURCE_FILL | DKV_POLICY_KV_DESCRIPTOR)))
    return DKV_ERR_INVALID;
  if (p->p != 1 && p->p != 2 && p->p != 4) return DKV_ERR_UNSUPPORTED;
  if (p->sigma2_log2 < -8 || p->sigma2_log2 > 16) return DKV_ERR_UNSUPPORTED;
  if (p->tau_log2_den < 0 || p->tau_log2_den > 8) return DKV_ERR_RANGE;
  if (p->tau_num < 1 || p->tau_num > (1 << 16)) return DKV_ERR_RANGE;
  if (p->tau_num <= (1 << p->tau_log2_den)) return DKV_ERR_RANGE;  // tau > 1
  if (p->delta_q < 1 || p->delta_q > (int64_t(1) << 40)) return DKV_ERR_RANGE;
  out->inv_sigma2 = ldexpf(1.0f, -p->sigma2_log2);
  out->p = p->p;
  out->tau_num = p->tau_num;
  out->tau_shift = p->tau_log2_den;
  out->delta_q = p->delta_q;
  out->block_id = block_id;
  out->flags = p->flags;
  return DKV_OK;
}

// The [K; V] retention geometry runs on the bf16 MFMA path and reads the
// candidates' values.
int check_geometry(const dkv_bank *bk, const dkv_segment *seg, const Prm &p) {
  if (p.flags & DKV_POLICY_SEQUENTIAL) {
    if (bk->dtype != DKV_BF16) return DKV_ERR_UNSUPPORTED;
    if (bk->group_size > kSeqMaxGroup) return DKV_ERR_SHAPE;
  }
  if (!(p.flags & DKV_POLICY_KV_DESCRIPTOR)) return DKV_OK;
  if (bk->dtype != DKV_BF16) return DKV_ERR_UNSUPPORTED;
  if (seg->n > 0 && !seg->v) return DKV_ERR_INVALID;
  return DKV_OK;
}

// Scratch of densitykv_update_bank_noalloc: a static device array, one copy per
// device (the runtime places it with the code object), so that call allocates
// nothing.  Host code never uses the array's name as an address: the device
// address comes from hipGetSymbolAddress with that device current and is kept
// per device.
static __device__ __align__(256) unsigned char scratch[DKV_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices];

int current_device_scratch(void **ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return DKV_ERR_HIP;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return DKV_ERR_HIP;
    scratch_ptr[dev] = p;
  }
  *ptr = scratch_ptr[dev];
  return DKV_OK;
}

Geom geom_of(const dkv_bank *bk, int n) {
  Geom g;
  g.B = bk->num_banks;
  g.gs = bk->group_size;
  g.G = bk->num_banks / bk->group_size;
  g.d = bk->head_dim;
  g.Mcap = bk->capacity;
  g.N = n;
  g.dtype = bk->dtype;
  return g;
}

// Groups per batch of the sequential competition: as many whole groups as
// DKV_SEQ_WEIGHT_BYTES of pairwise weights hold, at least one, at most all.
int seq_default_groups(const dkv_bank *bank, int n) {
  const int G = bank->num_banks / bank->group_size;
  const size_t per = seq_group_weight_bytes(bank->group_size, bank->capacity, n);
  const size_t fit = per > 0 ? DKV_SEQ_WEIGHT_BYTES / per : (size_t)G;
  return (int)(fit < 1 ? 1 : (fit > (size_t)G ? (size_t)G : fit));
}

// The workspace layout of an update on `bytes` of workspace: with the
// sequential competition, the weight area takes as many whole groups as the
// bytes beyond the fixed part hold (at most all); 0 groups when not even one
// fits.  Returns the bytes the layout needs (with at least one group).
size_t update_layout(const dkv_bank *bank, int n, bool seq, size_t bytes, char *base, Workspace *ws) {
  const int B = bank->num_banks, G = B / bank->group_size;
  if (!seq)
    return workspace_layout(B, G, bank->capacity, n, bank->head_dim, ws, base);
  const size_t fixed = workspace_layout(B, G, bank->capacity, n, bank->head_dim, nullptr, nullptr, true, 0);
  const size_t per = seq_group_weight_bytes(bank->group_size, bank->capacity, n);
  size_t groups = bytes > fixed ? (per > 0 ? (bytes - fixed) / per : (size_t)G) : 0;
  if (groups > (size_t)G) groups = (size_t)G;
  workspace_layout(B, G, bank->capacity, n, bank->head_dim, ws, base, true, (int)groups);
  return fixed + per;
}

}  // namespace

extern "C" {

int densitykv_workspace_size(const dkv_bank *bank, int32_t n_cand, size_t *bytes) {
  int rc = check_bank(bank);
  if (rc) return rc;
  if (!bytes) return DKV_ERR_INVALID;
  if (n_cand < 0 || n_cand > DKV_MAX_CANDIDATES) return DKV_ERR_SHAPE;
  *bytes = workspace_layout(bank->num_banks, bank->num_banks / bank->group_size, bank->capacity, n_cand,
                            bank->head_dim, nullptr, nullptr);
  return DKV_OK;
}

int densitykv_workspace_size_policy(const dkv_bank *bank, int32_t n_cand, uint32_t flags, size_t *bytes) {
  int rc = check_bank(bank);
  if (rc) return rc;
  if (!bytes) return DKV_ERR_INVALID;
  if (n_cand < 0 || n_cand > DKV_MAX_CANDIDATES) return DKV_ERR_SHAPE;
  const bool seq = (flags & DKV_POLICY_SEQUENTIAL) != 0;
  *bytes = workspace_layout(bank->num_banks, bank->num_banks / bank->group_size, bank->capacity, n_cand,
                            bank->head_dim, nullptr, nullptr, seq, seq ? seq_default_groups(bank, n_cand) : 0);
  return DKV_OK;
}

int densitykv_score(const dkv_bank *bank, const dkv_segment *seg, const dkv_params *prm,
                    int64_t *cand_score_q, float *cand_score_f32, int64_t *bank_density_q,
                    void *workspace, size_t workspace_bytes, void *stream) {
  int rc = check_bank(bank);
  if (!rc) rc = check_segment(seg);
  Prm p{};
  if (!rc) rc = check_params(prm, &p, seg->block_id);
  if (!rc) rc = check_geometry(bank, seg, p);
  if (rc) return rc;
  Workspace ws{};
  const size_t need = workspace_layout(bank->num_banks, bank->num_banks / bank->group_size, bank->capacity,
                                       seg->n, bank->head_dim, &ws, static_cast<char *>(workspace));
  if (!workspace || workspace_bytes < need) return DKV_ERR_WORKSPACE;
  const Geom g = geom_of(bank, seg->n);
  hipError_t e = launch_score(*bank, *seg, g, p, cand_score_q, cand_score_f32, bank_density_q, ws,
                              static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}

int densitykv_update_bank(dkv_bank *bank, const dkv_segment *seg, const dkv_params *prm, dkv_update_out *out,
                          void *workspace, size_t workspace_bytes, void *stream) {
  int rc = check_bank(bank);
  if (!rc) rc = check_segment(seg);
  Prm p{};
  if (!rc) rc = check_params(prm, &p, seg->block_id);
  if (!rc) rc = check_geometry(bank, seg, p);
  if (rc) return rc;
  Workspace ws{};
  const size_t need = update_layout(bank, seg->n, (p.flags & DKV_POLICY_SEQUENTIAL) != 0, workspace_bytes,
                                    static_cast<char *>(workspace), &ws);
  if (!workspace || workspace_bytes < need) return DKV_ERR_WORKSPACE;
  const Geom g = geom_of(bank, seg->n);
  hipError_t e = launch_update(*bank, *seg, g, p, out, ws, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}

int densitykv_update_bank_noalloc(dkv_bank *bank, const dkv_segment *seg, const dkv_params *prm,
                                  dkv_update_out *out, void *stream) {
  int rc = check_bank(bank);
  if (!rc) rc = check_segment(seg);
  Prm p{};
  if (!rc) rc = check_params(prm, &p, seg->block_id);
  if (!rc) rc = check_geometry(bank, seg, p);
  if (rc) return rc;
  const size_t need = update_layout(bank, seg->n, (p.flags & DKV_POLICY_SEQUENTIAL) != 0, 0, nullptr, nullptr);
  if (need > DKV_NOALLOC_SCRATCH_BYTES) return DKV_ERR_SCRATCH;
  void *ws = nullptr;
  rc = current_device_scratch(&ws);
  if (rc) return rc;
  return densitykv_update_bank(bank, seg, prm, out, ws, DKV_NOALLOC_SCRATCH_BYTES, stream);
}

int densitykv_bank_attention_sink(const dkv_bank *bank, const void *q, int32_t n_query, const void *sink_k,
                                  const void *sink_v, int32_t n_sink, const void *win_k, const void *win_v,
                                  int32_t n_window, void *out, float softmax_scale, void *stream) {
  int rc = check_bank(bank);
  if (rc) return rc;
  if (n_query < 0 || n_window < 0 || n_sink < 0 || n_query > (1 << 24) || n_window > (1 << 24) ||
      n_sink > (1 << 24))
    return DKV_ERR_SHAPE;
  if (n_query > 0 && (!q || !out)) return DKV_ERR_INVALID;
  if (n_window > 0 && (!win_k || !win_v)) return DKV_ERR_INVALID;
  if (n_sink > 0 && (!sink_k || !sink_v)) return DKV_ERR_INVALID;
  if (!(softmax_scale > 0.0f) || softmax_scale > 1e6f) return DKV_ERR_RANGE;
  const Geom g = geom_of(bank, 0);
  hipError_t e = launch_attention(*bank, q, n_query, KvSeg{win_k, win_v, n_window}, KvSeg{sink_k, sink_v, n_sink},
                                  out, softmax_scale, g, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}

int densitykv_bank_attention(const dkv_bank *bank, const void *q, int32_t n_query, const void *win_k,
                             const void *win_v, int32_t n_window, void *out, float softmax_scale,
                             void *stream) {
  return densitykv_bank_attention_sink(bank, q, n_query, nullptr, nullptr, 0, win_k, win_v, n_window, out,
                                       softmax_scale, stream);
}

int densitykv_pair_weight_q23(const float *d2, int64_t n, const dkv_params *prm, int32_t *w_q23,
                              void *stream) {
  Prm p{};
  int rc = check_params(prm, &p, 0);
  if (rc) return rc;
  if (n < 0) return DKV_ERR_SHAPE;
  if (n > 0 && (!d2 || !w_q23)) return DKV_ERR_INVALID;
  hipError_t e = launch_pair_weight(d2, n, p, w_q23, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? DKV_OK : DKV_ERR_HIP;
}

const char *densitykv_status_string(int status) {
  switch (status) {
    case DKV_OK: return "ok";
    case DKV_ERR_INVALID: return "invalid argument";
    case DKV_ERR_SHAPE: return "shape or size out of range";
    case DKV_ERR_UNSUPPORTED: return "unsupported head_dim, p or sigma^2";
    case DKV_ERR_WORKSPACE: return "workspace missing or too small";
    case DKV_ERR_RANGE: return "parameter out of fixed-point range";
    case DKV_ERR_HIP: return "HIP launch error";
    case DKV_ERR_SCRATCH: return "update needs more than the static scratch of the no-allocation entry point";
    default: return "unknown status";
  }
}

}  // extern "C"
