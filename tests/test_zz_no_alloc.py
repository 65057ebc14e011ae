"""densitykv_update_bank_noalloc against densitykv_update_bank (needs an MI355X).

The no-allocation entry point runs the same kernels with the library's static
device scratch as workspace.  Two calls in a row, the second on a smaller
input (fewer banks, a smaller capacity and fewer candidates, so the scratch
still holds the first call's larger layout), must leave every bank array and
every output bit-identical to the update with a caller-provided workspace.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from gpu_util import dev  # noqa: E402
from paper_2608_27922_amd import api, synth  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.lib()


BANK_FIELDS = ("k", "v", "knorm", "rho", "base", "prov", "occupancy")
OUT_FIELDS = ("r_star", "n_admitted", "n_evicted", "admitted", "evicted", "order", "score_q", "first_cross",
              "rho_tilde")


def _blocks(B, Mcap, N, d, seed):
    rng = np.random.default_rng(seed)
    first = synth.random_grid_keys(rng, (B, Mcap, d), scale=0.3)
    second = synth.random_grid_keys(rng, (B, N, d), scale=0.3)
    # near-duplicates of the first block, so that the second update evicts
    k = N // 3
    second[:, :k] = synth.snap_keys(first[:, :k] + 0.02 * rng.standard_normal((B, k, d)))
    out = []
    for K in (first, second):
        V = rng.standard_normal(K.shape).astype(np.float32)
        out.append((dev(K, "bf16"), dev(V, "bf16")))
    return out


def _compare(B, Mcap, N, d, gs, seed, ctx):
    prm = api.Params(sigma2_log2=6 if d == 128 else 5)
    blocks = _blocks(B, Mcap, N, d, seed)
    ref = api.Bank(B, Mcap, d, dtype=torch.bfloat16, group_size=gs)
    got = api.Bank(B, Mcap, d, dtype=torch.bfloat16, group_size=gs)
    for t, (K, V) in enumerate(blocks):
        n = K.shape[1]
        o_ref = api.UpdateOut(ref, n, trace=True)
        o_got = api.UpdateOut(got, n, trace=True)
        api.update_bank(ref, K, V, t, prm, workspace=api.alloc_workspace(ref, n), out=o_ref)
        api.update_bank_noalloc(got, K, V, t, prm, out=o_got)
        torch.cuda.synchronize()
        for f in BANK_FIELDS:
            assert torch.equal(getattr(ref, f), getattr(got, f)), f"{ctx} block {t}: bank {f} differs"
        for f in OUT_FIELDS:
            assert torch.equal(getattr(o_ref, f), getattr(o_got, f)), f"{ctx} block {t}: output {f} differs"
    assert int(ref.occupancy.min()) > 0
    return int(o_ref.r_star.max()), int(o_ref.n_evicted.max())


def test_noalloc_matches_workspace_update_twice_shrinking():
    print("noalloc: call 1 (12 banks, capacity 4,680, 4,680 candidates)", flush=True)
    r1, e1 = _compare(12, 4680, 4680, 128, 12, 7, "large")
    print(f"noalloc: call 1 ok (r* {r1}, max evicted {e1}); call 2 (4 banks, capacity 700, 300 candidates)",
          flush=True)
    r2, e2 = _compare(4, 700, 300, 128, 2, 8, "small")
    print(f"noalloc: call 2 ok (r* {r2}, max evicted {e2})", flush=True)
    assert e1 > 0 and e2 > 0


def test_noalloc_rejects_oversize_before_launch():
    bank = api.Bank(360, 4680, 128, dtype=torch.bfloat16, group_size=12)
    K = torch.zeros(360, 4680, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(api.DkvError) as ei:
        api.update_bank_noalloc(bank, K, K, 0, api.Params())
    assert ei.value.status == -7
    assert int(bank.occupancy.abs().sum()) == 0
