"""Thin ctypes binding of libdensitykv.so (include/densitykv.h), same entry-point names.

Argument marshalling only: torch tensors supply device memory and the current
HIP stream; every step of the hot path runs in the library's kernels.  There is
no fallback: if the library has not been built, loading raises.

Typical use (bf16 banks, one layer of 12 heads sharing the admitted prefix):

    bank = Bank(12, 4680, 128, dtype=torch.bfloat16, group_size=12)
    prm = Params(sigma2_log2=6)                      # sigma^2 = 64, p = 2, tau = 2
    ws = alloc_workspace(bank, 4680, prm.flags)      # reuse across updates
    out = UpdateOut(bank, 4680)                      # r*, admitted / evicted lists
    update_bank(bank, seg_k, seg_v, block_id, prm, workspace=ws, out=out)
    o = bank_attention(bank, q, win_k, win_v)        # queries over bank + window

Policy variants are Params.flags bits (POLICY_*); the sequential competition
needs the larger workspace that alloc_workspace(bank, n, flags) sizes.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdensitykv.so")

DKV_BF16, DKV_F32 = 0, 1
MAX_CANDIDATES, MAX_CAPACITY, MAX_BLOCK_ID = 8191, 32767, 16777215
# dkv_params.flags: policy ablations of Table 1(b) (0 = the paper's policy)
POLICY_SOURCE_ORDER = 0x1   # prefixes in source order instead of score order
POLICY_REFRESH_BASE = 0x2   # b = max(rho, delta) for every retained state after the update
POLICY_DENSEST_ONLY = 0x4   # no mandatory set: release the e densest states
POLICY_SOURCE_FILL = 0x8    # violators, then fill in admission order
POLICY_KV_DESCRIPTOR = 0x10  # densities on the concatenated [k; v] rows (bf16 banks; values on the key grid)
POLICY_SEQUENTIAL = 0x20    # within-block sequential competition (bf16 banks; larger workspace)

# Bytes of the static device scratch behind update_bank_noalloc (DKV_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 64 << 20
SEQ_WEIGHT_BYTES = 32 << 30     # pairwise-weight bytes the sequential workspace size is sized for

ENTRY_POINTS = ("densitykv_workspace_size", "densitykv_workspace_size_policy", "densitykv_score",
                "densitykv_update_bank", "densitykv_update_bank_noalloc",
                "densitykv_bank_attention", "densitykv_bank_attention_sink", "densitykv_pair_weight_q23",
                "densitykv_status_string")

_vp = ctypes.c_void_p


class DkvBank(ctypes.Structure):
    _fields_ = [("num_banks", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("k", _vp), ("v", _vp), ("knorm", _vp), ("rho", _vp),
                ("base", _vp), ("prov", _vp), ("occupancy", _vp), ("budget", _vp)]


class DkvSegment(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("block_id", ctypes.c_int32), ("k", _vp), ("v", _vp)]


class DkvParams(ctypes.Structure):
    _fields_ = [("sigma2_log2", ctypes.c_int32), ("p", ctypes.c_int32), ("tau_num", ctypes.c_int32),
                ("tau_log2_den", ctypes.c_int32), ("delta_q", ctypes.c_int64), ("flags", ctypes.c_uint32)]


class DkvUpdateOut(ctypes.Structure):
    _fields_ = [("r_star", _vp), ("n_admitted", _vp), ("n_evicted", _vp), ("admitted", _vp),
                ("evicted", _vp), ("order", _vp), ("score_q", _vp), ("first_cross", _vp),
                ("rho_tilde", _vp)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_27922_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.densitykv_workspace_size.argtypes = [P(DkvBank), ctypes.c_int32, P(ctypes.c_size_t)]
        L.densitykv_workspace_size_policy.argtypes = [P(DkvBank), ctypes.c_int32, ctypes.c_uint32,
                                                      P(ctypes.c_size_t)]
        L.densitykv_score.argtypes = [P(DkvBank), P(DkvSegment), P(DkvParams), _vp, _vp, _vp, _vp,
                                      ctypes.c_size_t, _vp]
        L.densitykv_update_bank.argtypes = [P(DkvBank), P(DkvSegment), P(DkvParams), P(DkvUpdateOut), _vp,
                                            ctypes.c_size_t, _vp]
        L.densitykv_update_bank_noalloc.argtypes = [P(DkvBank), P(DkvSegment), P(DkvParams), P(DkvUpdateOut),
                                                    _vp]
        L.densitykv_bank_attention.argtypes = [P(DkvBank), _vp, ctypes.c_int32, _vp, _vp, ctypes.c_int32, _vp,
                                               ctypes.c_float, _vp]
        L.densitykv_bank_attention_sink.argtypes = [P(DkvBank), _vp, ctypes.c_int32, _vp, _vp, ctypes.c_int32,
                                                    _vp, _vp, ctypes.c_int32, _vp, ctypes.c_float, _vp]
        L.densitykv_pair_weight_q23.argtypes = [_vp, ctypes.c_int64, P(DkvParams), _vp, _vp]
        L.densitykv_status_string.argtypes = [ctypes.c_int]
        L.densitykv_status_string.restype = ctypes.c_char_p
        for name in ENTRY_POINTS[:-1]:
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


class DkvError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib().densitykv_status_string(status).decode()} ({status})")


def _check(status: int, where: str):
    if status != 0:
        raise DkvError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


@dataclass(frozen=True)
class Params:
    """Method parameters (defaults: sigma = 8 -> sigma^2 = 2^6, p = 2, tau = 2, delta = 1e-6)."""

    sigma2_log2: int = 6
    p: int = 2
    tau_num: int = 2
    tau_log2_den: int = 0
    delta_q: int = 8
    flags: int = 0

    def c(self) -> DkvParams:
        return DkvParams(self.sigma2_log2, self.p, self.tau_num, self.tau_log2_den, self.delta_q, self.flags)


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return DKV_BF16
    if dt == torch.float32:
        return DKV_F32
    raise ValueError(f"unsupported dtype {dt}")


class Bank:
    """Device state of B = num_banks (layer, head) banks, row stride `capacity`.

    All state tensors are views into one device allocation (256-byte aligned
    sections), so a whole-bank checkpoint is a single copy (snapshot/restore)."""

    _FIELDS = ("k", "v", "knorm", "rho", "base", "prov", "occupancy", "budget")

    def __init__(self, num_banks: int, capacity: int, head_dim: int, dtype=torch.bfloat16,
                 group_size: int = 1, budget=None, device="cuda"):
        self.B, self.Mcap, self.d, self.gs = num_banks, capacity, head_dim, group_size
        self.dtype = dtype
        dev = torch.device(device)
        B, M, d = num_banks, capacity, head_dim
        layout = [("k", dtype, (B, M, d)), ("v", dtype, (B, M, d)), ("knorm", torch.float32, (B, M)),
                  ("rho", torch.int64, (B, M)), ("base", torch.int64, (B, M)), ("prov", torch.int64, (B, M)),
                  ("occupancy", torch.int32, (B,)), ("budget", torch.int32, (B,))]
        offs, total = [], 0
        for name, dt, shape in layout:
            nbytes = torch.empty((), dtype=dt).element_size()
            for x in shape:
                nbytes *= x
            offs.append((name, dt, shape, total, nbytes))
            total += (nbytes + 255) // 256 * 256
        self._buf = torch.zeros(max(total, 256), dtype=torch.uint8, device=dev)
        for name, dt, shape, off, nbytes in offs:
            setattr(self, name, self._buf[off:off + nbytes].view(dt).view(shape))
        if budget is None:
            self.budget.fill_(capacity)
        else:
            self.budget.copy_(torch.as_tensor(budget, dtype=torch.int32))

    def c(self) -> DkvBank:
        return DkvBank(self.B, self.gs, self.d, self.Mcap, _dtype_code(self.dtype), self.k.data_ptr(),
                       self.v.data_ptr(), self.knorm.data_ptr(), self.rho.data_ptr(), self.base.data_ptr(),
                       self.prov.data_ptr(), self.occupancy.data_ptr(), self.budget.data_ptr())

    def state_dict(self):
        """Checkpoint of the bank state, one cloned device tensor per field."""
        return {n: getattr(self, n).clone() for n in self._FIELDS}

    def load_state_dict(self, sd):
        for n, t in sd.items():
            getattr(self, n).copy_(t)

    def snapshot(self) -> torch.Tensor:
        """Checkpoint of the whole bank state as one device buffer."""
        return self._buf.clone()

    def restore(self, snap: torch.Tensor):
        """Restore a snapshot() of this bank (one device-to-device copy on the current stream)."""
        self._buf.copy_(snap)


def workspace_size(bank: Bank, n_cand: int, flags: int = 0) -> int:
    """densitykv_workspace_size, or densitykv_workspace_size_policy for non-zero flags."""
    out = ctypes.c_size_t(0)
    cb = bank.c()
    if flags:
        _check(lib().densitykv_workspace_size_policy(ctypes.byref(cb), int(n_cand), int(flags), ctypes.byref(out)),
               "workspace_size_policy")
    else:
        _check(lib().densitykv_workspace_size(ctypes.byref(cb), int(n_cand), ctypes.byref(out)), "workspace_size")
    return int(out.value)


def seq_group_weight_bytes(bank: Bank, n_cand: int) -> int:
    """Pairwise-weight bytes of one group in the sequential competition."""
    L = bank.Mcap + max(int(n_cand), 0)
    return bank.gs * L * L * 4


def alloc_workspace(bank: Bank, n_cand: int, flags: int = 0, seq_groups: Optional[int] = None) -> torch.Tensor:
    """Workspace of densitykv_workspace_size_policy; with POLICY_SEQUENTIAL and
    `seq_groups`, room for the pairwise weights of that many groups instead
    (the update then walks that many groups at a time)."""
    size = workspace_size(bank, n_cand, flags)
    if seq_groups is not None and flags & POLICY_SEQUENTIAL:
        per, G = seq_group_weight_bytes(bank, n_cand), bank.B // bank.gs
        default = min(G, max(1, SEQ_WEIGHT_BYTES // per))
        size += (min(max(int(seq_groups), 1), G) - default) * per
    return torch.empty(size, dtype=torch.uint8, device=bank.k.device)


def _segment(seg_k: Optional[torch.Tensor], seg_v: Optional[torch.Tensor], n: int, block_id: int):
    return DkvSegment(int(n), int(block_id), None if seg_k is None else seg_k.data_ptr(),
                      None if seg_v is None else seg_v.data_ptr())


def _check_seg(bank: Bank, seg_k, seg_v):
    if seg_k is None:
        return 0
    if seg_k.dim() != 3 or seg_k.shape[0] != bank.B or seg_k.shape[2] != bank.d:
        raise ValueError("segment keys must be [num_banks, n, head_dim]")
    if seg_v is None or seg_v.shape != seg_k.shape:
        raise ValueError("segment values must match the keys' shape")
    for t in (seg_k, seg_v):
        if t.dtype != bank.dtype or not t.is_contiguous() or t.device != bank.k.device:
            raise ValueError("segment tensors must be contiguous, on the bank's device, in the bank dtype")
    return int(seg_k.shape[1])


def score(bank: Bank, seg_k: torch.Tensor, seg_v: torch.Tensor, params: Params = Params(),
          want_q=True, want_f32=True, want_density=False, workspace: Optional[torch.Tensor] = None):
    """densitykv_score: returns (score_q [B,N] int64 | None, score_f32 [B,N] | None, density [B,Mcap] | None)."""
    n = _check_seg(bank, seg_k, seg_v)
    dev = bank.k.device
    sq = torch.zeros(bank.B, n, dtype=torch.int64, device=dev) if want_q else None
    sf = torch.zeros(bank.B, n, dtype=torch.float32, device=dev) if want_f32 else None
    dens = torch.zeros(bank.B, bank.Mcap, dtype=torch.int64, device=dev) if want_density else None
    ws = workspace if workspace is not None else alloc_workspace(bank, n, params.flags)
    cb, cs, cp = bank.c(), _segment(seg_k, seg_v, n, 0), params.c()
    _check(lib().densitykv_score(ctypes.byref(cb), ctypes.byref(cs), ctypes.byref(cp), _ptr(sq), _ptr(sf),
                                 _ptr(dens), _ptr(ws), ws.numel(), _stream()), "score")
    return sq, sf, dens


class UpdateOut:
    """Optional device outputs of one update (allocated on request)."""

    def __init__(self, bank: Bank, n: int, trace: bool = False):
        dev, B = bank.k.device, bank.B
        G = B // bank.gs
        i32 = dict(dtype=torch.int32, device=dev)
        self.r_star = torch.zeros(G, **i32)
        self.n_admitted = torch.zeros(B, **i32)
        self.n_evicted = torch.zeros(B, **i32)
        self.admitted = torch.zeros(B, max(n, 1), **i32)
        self.evicted = torch.zeros(B, bank.Mcap, **i32)
        self.order = torch.zeros(B, max(n, 1), **i32) if trace else None
        self.score_q = torch.zeros(B, max(n, 1), dtype=torch.int64, device=dev) if trace else None
        self.first_cross = torch.full((B, bank.Mcap), -1, **i32) if trace else None
        self.rho_tilde = torch.zeros(B, bank.Mcap, dtype=torch.int64, device=dev) if trace else None

    def c(self) -> DkvUpdateOut:
        f = lambda t: None if t is None else t.data_ptr()
        return DkvUpdateOut(f(self.r_star), f(self.n_admitted), f(self.n_evicted), f(self.admitted),
                            f(self.evicted), f(self.order), f(self.score_q), f(self.first_cross),
                            f(self.rho_tilde))

    def walk_ok(self) -> bool:
        """False when a group's sequential walk gave up waiting (r_star = -1);
        synchronizes with the device."""
        return bool(torch.all(self.r_star >= 0).item())


class _StepCounts(UpdateOut):
    """r_star alone: what the sequential competition always returns, so that a
    walk that gave up (r_star = -1) can be seen after the call."""

    def __init__(self, bank: Bank):
        self.r_star = torch.zeros(bank.B // bank.gs, dtype=torch.int32, device=bank.k.device)
        self.n_admitted = self.n_evicted = self.admitted = self.evicted = None
        self.order = self.score_q = self.first_cross = self.rho_tilde = None


def _outputs(bank: Bank, params: "Params", out):
    if out is None and params.flags & POLICY_SEQUENTIAL:
        return _StepCounts(bank)
    return out


def update_bank(bank: Bank, seg_k: Optional[torch.Tensor], seg_v: Optional[torch.Tensor], block_id: int,
                params: Params = Params(), workspace: Optional[torch.Tensor] = None,
                out: Optional[UpdateOut] = None) -> Optional[UpdateOut]:
    """densitykv_update_bank: updates `bank` in place on the current stream.
    With POLICY_SEQUENTIAL and no `out`, returns an output object holding
    r_star only (check it with walk_ok() once the stream has run)."""
    n = _check_seg(bank, seg_k, seg_v)
    ws = workspace if workspace is not None else alloc_workspace(bank, n, params.flags)
    out = _outputs(bank, params, out)
    cb, cs, cp = bank.c(), _segment(seg_k, seg_v, n, block_id), params.c()
    co = out.c() if out is not None else None
    _check(lib().densitykv_update_bank(ctypes.byref(cb), ctypes.byref(cs), ctypes.byref(cp),
                                       ctypes.byref(co) if co is not None else None, _ptr(ws), ws.numel(),
                                       _stream()), "update_bank")
    return out


def update_bank_noalloc(bank: Bank, seg_k: Optional[torch.Tensor], seg_v: Optional[torch.Tensor], block_id: int,
                        params: Params = Params(), out: Optional[UpdateOut] = None) -> Optional[UpdateOut]:
    """densitykv_update_bank_noalloc: the same update with the library's static
    device scratch as workspace (no allocation by the call; sizes whose workspace
    exceeds NOALLOC_SCRATCH_BYTES raise DkvError)."""
    n = _check_seg(bank, seg_k, seg_v)
    out = _outputs(bank, params, out)
    cb, cs, cp = bank.c(), _segment(seg_k, seg_v, n, block_id), params.c()
    co = out.c() if out is not None else None
    _check(lib().densitykv_update_bank_noalloc(ctypes.byref(cb), ctypes.byref(cs), ctypes.byref(cp),
                                               ctypes.byref(co) if co is not None else None, _stream()),
           "update_bank_noalloc")
    return out


def _kv_segment(bank: Bank, k: Optional[torch.Tensor], v: Optional[torch.Tensor], what: str) -> int:
    if k is None:
        return 0
    if k.dim() != 3 or k.shape[0] != bank.B or k.shape[2] != bank.d or v is None or v.shape != k.shape:
        raise ValueError(f"{what} must be [num_banks, n, head_dim] keys and values")
    if not (k.is_contiguous() and v.is_contiguous()) or k.dtype != bank.dtype or v.dtype != bank.dtype:
        raise ValueError(f"{what} tensors must be contiguous in the bank dtype")
    return int(k.shape[1])


def _check_q(bank: Bank, q: torch.Tensor):
    if q.dim() != 3 or q.shape[0] != bank.B or q.shape[2] != bank.d or q.dtype != bank.dtype or not q.is_contiguous():
        raise ValueError("q must be a contiguous [num_banks, n_query, head_dim] tensor in the bank dtype")


def bank_attention(bank: Bank, q: torch.Tensor, win_k: Optional[torch.Tensor], win_v: Optional[torch.Tensor],
                   softmax_scale: Optional[float] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """densitykv_bank_attention: softmax(q [bank; window]^T * scale) [bank; window]."""
    _check_q(bank, q)
    nw = _kv_segment(bank, win_k, win_v, "window")
    if out is None:
        out = torch.empty_like(q)
    scale = (1.0 / bank.d ** 0.5) if softmax_scale is None else float(softmax_scale)
    cb = bank.c()
    _check(lib().densitykv_bank_attention(ctypes.byref(cb), _ptr(q), int(q.shape[1]), _ptr(win_k), _ptr(win_v),
                                          nw, _ptr(out), ctypes.c_float(scale), _stream()), "bank_attention")
    return out


def bank_attention_sink(bank: Bank, q: torch.Tensor, sink_k: Optional[torch.Tensor], sink_v: Optional[torch.Tensor],
                        win_k: Optional[torch.Tensor], win_v: Optional[torch.Tensor],
                        softmax_scale: Optional[float] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """densitykv_bank_attention_sink: softmax over [bank; window; sink]."""
    _check_q(bank, q)
    ns = _kv_segment(bank, sink_k, sink_v, "sink")
    nw = _kv_segment(bank, win_k, win_v, "window")
    if out is None:
        out = torch.empty_like(q)
    scale = (1.0 / bank.d ** 0.5) if softmax_scale is None else float(softmax_scale)
    cb = bank.c()
    _check(lib().densitykv_bank_attention_sink(ctypes.byref(cb), _ptr(q), int(q.shape[1]), _ptr(sink_k),
                                               _ptr(sink_v), ns, _ptr(win_k), _ptr(win_v), nw, _ptr(out),
                                               ctypes.c_float(scale), _stream()), "bank_attention_sink")
    return out


def pair_weight_q23(d2: torch.Tensor, params: Params = Params()) -> torch.Tensor:
    """densitykv_pair_weight_q23 over a float32 device tensor of squared distances."""
    d2 = d2.contiguous()
    w = torch.empty(d2.shape, dtype=torch.int32, device=d2.device)
    cp = params.c()
    _check(lib().densitykv_pair_weight_q23(_ptr(d2), d2.numel(), ctypes.byref(cp), _ptr(w), _stream()),
           "pair_weight_q23")
    return w
