"""Group advantages (Eq. 2) of kept training groups on the GPU against the
oracle: random groups at the selection sweep's size (4096 groups of k = 8),
edge cases (incomplete groups, equal rewards, k = 1 and k = 64), and the
kept sets of a real rollout."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle.advantage import group_advantages
from workload import get_config, rollout_inputs
from workload.gen import synthetic_rewards

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _b():
    from paper_2605_30859_amd import binding
    binding.load_library()
    return binding


def _check(kept, reward, eps=1e-6):
    B = _b()
    kd = torch.from_numpy(np.ascontiguousarray(kept, dtype=np.int32)).to(DEV)
    rd = torch.from_numpy(np.ascontiguousarray(reward, dtype=np.float32)).to(DEV)
    ad = torch.full(kd.shape, 7.0, dtype=torch.float32, device=DEV)
    B.darts_group_advantages(kd, rd, ad, eps)
    got = ad.cpu().numpy()
    for i, row in enumerate(kept):
        if (row < 0).any() or (row >= len(reward)).any():
            assert np.isnan(got[i]).all()
            continue
        exp = group_advantages([float(reward[g]) for g in row], eps)
        assert np.allclose(got[i], exp, rtol=0, atol=2e-5), (i, got[i], exp)
    return got


@pytest.mark.parametrize("kind", ["binary", "normal"])
def test_advantages_sweep_size(kind):
    rng = np.random.default_rng(5)
    n_groups, m, k = 4096, 16, 8
    kept = np.stack([i * m + rng.choice(m, k, replace=False) for i in range(n_groups)]).astype(np.int32)
    reward = synthetic_rewards(n_groups * m, 1) if kind == "binary" else \
        rng.normal(0, 3, n_groups * m).astype(np.float32)
    got = _check(kept, reward)
    assert np.abs(got.sum(axis=1)).max() < 1e-4


def test_advantages_edge_cases():
    rng = np.random.default_rng(6)
    reward = rng.normal(0, 1, 256).astype(np.float32)
    reward[:64] = 1.0
    kept = np.array([[0, 1, 2, 3], [5, -1, 7, 9], [10, 11, 12, 300], [64, 100, 3, 200]], np.int32)
    got = _check(kept, reward)
    assert (got[0] == 0).all()                                  # equal rewards
    _check(np.arange(256, dtype=np.int32).reshape(256, 1), reward)          # k = 1
    _check(np.arange(256, dtype=np.int32).reshape(4, 64), reward)           # k = 64
    B = _b()
    with pytest.raises(B.DartsError):
        B.darts_group_advantages(torch.zeros((1, 65), dtype=torch.int32, device=DEV),
                                 torch.zeros(65, device=DEV), torch.zeros((1, 65), device=DEV))


def test_advantages_of_rollout_kept_sets():
    B = _b()
    model, run = get_config("tiny")
    prompts, forced = rollout_inputs(model, run)
    ro = B.Rollout(model, run)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    ro.run_to_completion(pr, fl)
    kept = ro.kept.cpu().numpy()
    ro.close()
    assert (kept >= 0).all()
    _check(kept, synthetic_rewards(run.n_prompts * run.m, 3))
