"""Seeded synthetic inputs for the DensityKV hot path.

Stand-ins for the post-RoPE keys, values and queries that the paper's video
backbone (Wan2.1-T2V-1.3B: d_k = d_v = 128, 1,560 tokens per latent frame,
3-frame blocks of N = 4,680 candidates; Supp. D) would produce.  The module
only draws numbers: it holds none of the method's arithmetic and is the one
piece shared by the tests, the oracle runs and the benchmark.

Recipe (per (config, layer, head), independent NumPy PCG64 streams from base
seed 0, the paper's generation seed):
  * cluster centres c_j = g / |g| with g ~ N(0, I_d);
  * a token is c_z + 0.3 * eps, eps ~ N(0, I_d) per component, z uniform over
    the active clusters;
  * keys are snapped to the 1/64 grid, clip(rint(64 x), -127, 127) / 64, so
    that every key-key Gram is exact in fp32 (the contract that makes the
    oracle and the kernels agree bit for bit);
  * values and queries are fresh mixture draws rounded to the storage dtype.
Config specifics: near-duplicates of bank tokens (config 2), centre drift by
a 0.05 random-walk step per block (configs 3 and 5), 256 clusters with
16 active per block and a recurring active set every 10 blocks (config 4),
per-head budgets drawn from {2340, 4680, 9360, 18720} (config 5).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Optional, Tuple

import numpy as np

GRID = 64          # keys are integers / 64
GRID_MAX = 127     # |integer| <= 127


@dataclass(frozen=True)
class Config:
    seed_id: int               # seeds this workload's random streams
    name: str
    layers: int
    heads: int
    d: int
    dtype: str                 # "bf16" or "f32"
    n_cand: int                # N candidates per block
    n_query: int
    n_window: int
    budget: int                # per-head budget (max budget when ragged)
    clusters: int
    blocks: int                # number of updates in the run
    group_size: int            # heads sharing one admitted prefix length
    sigma2_log2: int           # sigma^2 = d_k / 2 (Supp. B bandwidth calibration)
    starts_full: bool = False  # bank built first from a block of `budget` tokens
    dup_frac: float = 0.0
    drift: float = 0.0
    active: int = 0            # active clusters per block (0: all)
    revisit: int = 0           # recurring active set period (0: none)
    ragged: Tuple[int, ...] = ()

    @property
    def banks(self) -> int:
        return self.layers * self.heads


WORKLOADS: Dict[str, Config] = {c.name: c for c in (
    # 1 layer x 2 heads, d 64, fp32, budget 256 (starts full), 64 candidates, 64 queries + 64 window
    Config(1, "tiny", 1, 2, 64, "f32", 64, 64, 64, 256, 8, 1, 2, 5, starts_full=True),
    # 1 layer x 12 heads, d 128, bf16, budget 4680 (starts full), 4680 candidates with 30%
    # near-duplicates, 4680 queries over bank + 4680 window
    Config(2, "single_layer", 1, 12, 128, "bf16", 4680, 4680, 4680, 4680, 64, 1, 12, 6,
           starts_full=True, dup_frac=0.3),
    # 30 layers x 12 heads, 20 blocks of 4680 into budget 9360, drifting centres
    Config(3, "rollout", 30, 12, 128, "bf16", 4680, 4680, 4680, 9360, 64, 20, 12, 6, drift=0.05),
    # 30 layers x 12 heads, 80 blocks into budget 18720, 256 clusters, recurring sets every 10 blocks
    Config(4, "long_rollout", 30, 12, 128, "bf16", 4680, 4680, 4680, 18720, 256, 80, 12, 6,
           active=16, revisit=10),
    # 30 layers x 12 heads, 160 blocks, per-head budgets from {2340, 4680, 9360, 18720}, heads independent
    Config(5, "headwise_budgets", 30, 12, 128, "bf16", 4680, 4680, 4680, 18720, 64, 160, 1, 6,
           drift=0.05, ragged=(2340, 4680, 9360, 18720)),
)}

ROLE_CENTRES, ROLE_K, ROLE_V, ROLE_Q, ROLE_DUP, ROLE_BUDGET, ROLE_DRIFT, ROLE_ACTIVE = range(8)


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, *key]))


def snap_keys(x: np.ndarray) -> np.ndarray:
    """Round to the 1/64 key grid (float32, exact in bf16)."""
    return (np.clip(np.rint(x * GRID), -GRID_MAX, GRID_MAX) / GRID).astype(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float values to the storage dtype, returned as float32 holding exact values."""
    x = np.asarray(x, np.float32)
    if dtype == "f32":
        return x
    if dtype != "bf16":
        raise ValueError(dtype)
    b = x.view(np.uint32).astype(np.uint64)
    rounded = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000  # round to nearest even
    return rounded.astype(np.uint32).view(np.float32)


def budgets(cfg: Config, seed: int = 0) -> np.ndarray:
    """Per-(layer, head) budgets, shape (layers * heads,)."""
    if not cfg.ragged:
        return np.full(cfg.banks, cfg.budget, np.int32)
    r = _rng(seed, cfg.seed_id, ROLE_BUDGET)
    return np.asarray(cfg.ragged, np.int32)[r.integers(0, len(cfg.ragged), cfg.banks)]


class HeadStream:
    """Seeded token source of one (config, layer, head).

    block(t) returns (K, V, Q) for block t: K, V with `n` rows, Q with
    cfg.n_query rows.  Blocks are indexed from 0; the drift state is advanced
    deterministically, so any block can be requested in any order."""

    def __init__(self, cfg: Config, layer: int, head: int, seed: int = 0):
        self.cfg, self.layer, self.head, self.seed = cfg, layer, head, seed
        r = _rng(seed, cfg.seed_id, layer, head, ROLE_CENTRES)
        g = r.standard_normal((cfg.clusters, cfg.d))
        self._c0 = g / np.linalg.norm(g, axis=1, keepdims=True)
        self._centres = {0: self._c0}
        self._dup_src: Optional[np.ndarray] = None

    def centres(self, t: int) -> np.ndarray:
        if self.cfg.drift == 0.0:
            return self._c0
        last = max(k for k in self._centres if k <= t)
        c = self._centres[last]
        for s in range(last + 1, t + 1):
            u = _rng(self.seed, self.cfg.seed_id, self.layer, self.head, ROLE_DRIFT, s).standard_normal(c.shape)
            u /= np.linalg.norm(u, axis=1, keepdims=True)
            c = c + self.cfg.drift * u
            c = c / np.linalg.norm(c, axis=1, keepdims=True)
            self._centres[s] = c
        return c

    def active_set(self, t: int) -> np.ndarray:
        cfg = self.cfg
        if cfg.active == 0:
            return np.arange(cfg.clusters)
        if cfg.revisit and t >= cfg.revisit and t % cfg.revisit == 0:
            return self.active_set(t - cfg.revisit)
        r = _rng(self.seed, cfg.seed_id, self.layer, self.head, ROLE_ACTIVE, t)
        return np.sort(r.choice(cfg.clusters, cfg.active, replace=False))

    def _mixture(self, role: int, t: int, n: int) -> np.ndarray:
        r = _rng(self.seed, self.cfg.seed_id, self.layer, self.head, role, t)
        act = self.active_set(t)
        z = act[r.integers(0, act.size, n)]
        noise = r.standard_normal((n, self.cfg.d), dtype=np.float32)
        return self.centres(t)[z].astype(np.float32) + np.float32(0.3) * noise

    def keys(self, t: int, n: int) -> np.ndarray:
        return snap_keys(self._mixture(ROLE_K, t, n))

    def values(self, t: int, n: int) -> np.ndarray:
        return to_storage(self._mixture(ROLE_V, t, n), self.cfg.dtype)

    def queries(self, t: int) -> np.ndarray:
        return to_storage(self._mixture(ROLE_Q, t, self.cfg.n_query), self.cfg.dtype)

    def near_duplicates(self, K: np.ndarray, bank_keys: np.ndarray, t: int) -> np.ndarray:
        """Replace a fraction cfg.dup_frac of the rows of K by near-duplicates
        (cosine > 0.95) of uniformly drawn rows of bank_keys."""
        cfg = self.cfg
        n = K.shape[0]
        r = _rng(self.seed, cfg.seed_id, self.layer, self.head, ROLE_DUP, t)
        k = int(round(cfg.dup_frac * n))
        rows = np.sort(r.choice(n, k, replace=False))
        src = r.integers(0, bank_keys.shape[0], k)
        out = K.copy()
        for i, s in zip(rows, src):
            base = bank_keys[s].astype(np.float64)
            while True:
                x = snap_keys(base + 0.05 * r.standard_normal(cfg.d))
                cos = float(x @ base) / (np.linalg.norm(x) * np.linalg.norm(base) + 1e-30)
                if cos > 0.95:
                    break
            out[i] = x
        return out


def single_update_case(cfg: Config, layer: int = 0, seed: int = 0, heads: Optional[range] = None):
    """Inputs of a starts-full configuration (configs 1 and 2) for one layer.

    Returns a dict of stacked float32 arrays over the layer's heads:
      init_K, init_V  (H, budget, d)  block 0: builds the full initial bank
      seg_K, seg_V    (H, N, d)       block 1: the incoming segment
      q               (H, Nq, d)      block 2 queries
      win_K, win_V    (H, W, d)       block 2 keys/values: the local window
    """
    heads = range(cfg.heads) if heads is None else heads
    out = {k: [] for k in ("init_K", "init_V", "seg_K", "seg_V", "q", "win_K", "win_V")}
    for h in heads:
        s = HeadStream(cfg, layer, h, seed)
        iK = s.keys(0, cfg.budget)
        out["init_K"].append(iK)
        out["init_V"].append(s.values(0, cfg.budget))
        sK = s.keys(1, cfg.n_cand)
        if cfg.dup_frac:
            sK = s.near_duplicates(sK, iK, 1)
        out["seg_K"].append(sK)
        out["seg_V"].append(s.values(1, cfg.n_cand))
        out["q"].append(s.queries(2))
        out["win_K"].append(s.keys(2, cfg.n_window))
        out["win_V"].append(s.values(2, cfg.n_window))
    return {k: np.stack(v) for k, v in out.items()}


def random_grid_keys(rng: np.random.Generator, shape, scale: float = 0.5) -> np.ndarray:
    """Generic grid keys for small tests (not a config workload)."""
    return snap_keys(scale * rng.standard_normal(shape))


def torch_layer_block(cfg: Config, layer: int, t: int, n: int, device, seed: int = 0):
    """Keys and values of one block for every head of one layer, drawn on the GPU.

    Same recipe as HeadStream (unit-norm centres fixed per (layer, head), tokens
    = centre + 0.3 N(0, I), keys snapped to the grid, values rounded to the
    storage dtype) from a seeded torch generator, without the drift / recurrence
    schedule.  Used to fill the layers that are not compared with the oracle in
    full-size runs, where generating 360 banks on the host would dominate."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed((seed * 1_000_003 + cfg.seed_id * 10_007 + layer) & 0x7FFFFFFF)
    H, d = cfg.heads, cfg.d
    c = torch.randn(H, cfg.clusters, d, generator=gen, device=device)
    c = c / c.norm(dim=-1, keepdim=True)
    gen.manual_seed((seed * 1_000_003 + cfg.seed_id * 10_007 + layer * 131 + 7 * t + 1) & 0x7FFFFFFF)
    out = []
    for _role in range(2):
        z = torch.randint(0, cfg.clusters, (H, n), generator=gen, device=device)
        x = torch.gather(c, 1, z[..., None].expand(H, n, d)) + 0.3 * torch.randn(H, n, d, generator=gen, device=device)
        out.append(x)
    k = (torch.clamp(torch.round(out[0] * GRID), -GRID_MAX, GRID_MAX) / GRID)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    return k.to(dt).contiguous(), out[1].to(dt).contiguous()


class TorchRollout:
    """Device-side draws of a rollout workload for every (layer, head) at once.

    The HeadStream recipe (unit-norm centres per (layer, head); tokens = centre
    + 0.3 N(0, I); keys snapped to the grid, values and queries rounded to the
    storage dtype; centre drift per block; active cluster sets with the
    recurring set) drawn from seeded torch generators on the device, so that a
    whole 360-bank run can be generated in HBM before it is timed.  Block t
    depends only on (seed, workload, t, role); the numbers differ from the
    NumPy streams, the distribution does not."""

    def __init__(self, cfg: Config, device, seed: int = 0):
        import torch
        self.torch, self.cfg, self.device, self.seed = torch, cfg, torch.device(device), seed
        self.B = cfg.layers * cfg.heads
        g = self._gen(ROLE_CENTRES, 0)
        c = torch.randn(self.B, cfg.clusters, cfg.d, generator=g, device=self.device)
        self._centres = {0: c / c.norm(dim=-1, keepdim=True)}

    def _gen(self, role: int, t: int):
        g = self.torch.Generator(device=self.device)
        g.manual_seed((((self.seed * 1_000_003 + self.cfg.seed_id) * 131 + role) * 100_003 + t) & 0x7FFFFFFFFFFF)
        return g

    def centres(self, t: int):
        cfg, torch = self.cfg, self.torch
        if cfg.drift == 0.0:
            return self._centres[0]
        last = max(k for k in self._centres if k <= t)
        c = self._centres[last]
        for s in range(last + 1, t + 1):
            u = torch.randn(c.shape, generator=self._gen(ROLE_DRIFT, s), device=self.device)
            c = c + cfg.drift * (u / u.norm(dim=-1, keepdim=True))
            c = c / c.norm(dim=-1, keepdim=True)
            self._centres[s] = c
        for k in [k for k in self._centres if 0 < k < t]:   # keep only what later blocks need
            del self._centres[k]
        return c

    def active_set(self, t: int):
        """[B, A] cluster indices active in block t."""
        cfg, torch = self.cfg, self.torch
        if cfg.active == 0:
            return torch.arange(cfg.clusters, device=self.device).expand(self.B, cfg.clusters)
        if cfg.revisit and t >= cfg.revisit and t % cfg.revisit == 0:
            return self.active_set(t - cfg.revisit)
        r = torch.rand(self.B, cfg.clusters, generator=self._gen(ROLE_ACTIVE, t), device=self.device)
        return r.argsort(dim=1)[:, :cfg.active]

    def _mixture(self, role: int, t: int, n: int):
        cfg, torch = self.cfg, self.torch
        g = self._gen(role, t)
        act = self.active_set(t)
        z = torch.gather(act, 1, torch.randint(0, act.shape[1], (self.B, n), generator=g, device=self.device))
        c = self.centres(t)
        x = torch.gather(c, 1, z[..., None].expand(self.B, n, cfg.d))
        return x.add_(torch.randn(self.B, n, cfg.d, generator=g, device=self.device), alpha=0.3)

    def _dtype(self):
        return self.torch.bfloat16 if self.cfg.dtype == "bf16" else self.torch.float32

    def keys(self, t: int, n: int):
        x = self._mixture(ROLE_K, t, n)
        return (self.torch.clamp(self.torch.round(x * GRID), -GRID_MAX, GRID_MAX) / GRID).to(self._dtype())

    def values(self, t: int, n: int):
        return self._mixture(ROLE_V, t, n).to(self._dtype())

    def queries(self, t: int):
        return self._mixture(ROLE_Q, t, self.cfg.n_query).to(self._dtype())
