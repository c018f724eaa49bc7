"""The long-tail rollout driver on the GPU (tiny bf16 model): every policy
runs its responses to completion, the cache length of every slot ends at
prompt + the tokens it emitted (AR caches one position per iteration, SD
n_emit), SD's block efficiency stays in [1, gamma + 1], and a rollout is
reproducible from its seeds."""
import numpy as np
import pytest

from gpu_common import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny_rollout():
    import torch
    from paper_2606_18967_amd import rollout
    torch.cuda.set_device(0)
    ro = rollout.Rollout(rollout.MODELS["TINY_BF16"], B=6, prompt=16, lmax=40, seed=5)
    yield ro
    ro.close()


@pytest.mark.parametrize("policy,gamma", [("ar", 5), ("sd", 5), ("sd", 11), ("toggle", 7), ("adaptive", 9)])
def test_tiny_rollout_completes_and_caches_every_emitted_token(tiny_rollout, policy, gamma):
    from paper_2606_18967_amd import sdrl
    ro = tiny_rollout
    L = np.array([3, 9, 1, 17, 5, 12])
    say(f"rollout policy={policy} gamma={gamma} lengths={L.tolist()}")
    cost = sdrl.cost_init(ro.cfg)               # the uncalibrated model: SD predicted to pay at this size
    res, st = ro.run(policy, gamma, 5.0, cost, 0.05, L, step=1)
    assert (st["gen"] >= L).all()
    kv = ro.kv_len.cpu().numpy()
    assert (kv - ro.prompt == st["gen"]).all()
    assert res.tokens == int(L.sum())
    if policy == "ar":
        assert res.ar_iters == L.max() and res.sd_iters == 0 and res.tau is None
    else:
        assert res.sd_iters >= 1 and 1.0 <= res.tau <= gamma + 1
        assert (st["gen"] - L <= gamma).all()            # at most gamma tokens past the end
    if policy in ("toggle", "adaptive"):
        assert res.switch_iter == 0 and res.switch_B == len(L)


def test_tiny_rollout_is_reproducible(tiny_rollout):
    from paper_2606_18967_amd import sdrl
    ro = tiny_rollout
    L = np.array([30, 2, 11, 7, 25, 19])
    cost = sdrl.cost_init(ro.cfg)
    say("rollout reproducibility (sd, gamma 5, twice)")
    a = ro.run("sd", 5, 5.0, cost, 0.05, L, step=3)
    b = ro.run("sd", 5, 5.0, cost, 0.05, L, step=3)
    assert (a[1]["gen"] == b[1]["gen"]).all()
    assert [t[4] for t in a[0].trace] == [t[4] for t in b[0].trace]
    c = ro.run("sd", 5, 5.0, cost, 0.05, L, step=4)               # another training step draws afresh
    assert c[0].tau is not None


@pytest.mark.parametrize("policy,gamma", [("ar", 5), ("sd", 5), ("toggle", 7)])
def test_graph_rollout_equals_padded_eager_rollout(policy, gamma):
    """The long-tail driver with per-(bucket, draft length) HIP graphs: live
    batches padded to buckets of 8 rows (spare slots carry the padding), each
    bucket's step captured once and replayed.  Every replay must give exactly
    the tokens of the same padded step run eagerly, and every live slot's
    cache length must end at prompt + the tokens it emitted."""
    import torch
    from paper_2606_18967_amd import rollout, sdrl
    torch.cuda.set_device(0)
    cfg = rollout.MODELS["TINY_BF16"]
    L = np.array([3, 30, 1, 17, 9, 12, 25, 5, 21, 14, 2])      # 11 sequences: buckets 16 and 8
    say(f"graph rollout policy={policy} gamma={gamma}")
    runs = []
    for graphs in (True, False):
        ro = rollout.Rollout(cfg, B=len(L), prompt=16, lmax=40, seed=9, graphs=graphs, padded=True)
        res, st = ro.run(policy, gamma, 5.0, sdrl.cost_init(ro.cfg), 0.05, L, step=2)
        kv = ro.kv_len[:ro.B].cpu().numpy()
        assert (kv - ro.prompt == st["gen"]).all()
        assert (st["gen"] >= L).all()
        runs.append((res, st))
        ro.close()
    (rg, sg), (re_, se) = runs
    assert (sg["gen"] == se["gen"]).all()
    assert [t[4] for t in rg.trace] == [t[4] for t in re_.trace]
    assert [t[:2] for t in rg.trace] == [t[:2] for t in re_.trace]
    assert rg.graphs >= 2 and re_.graphs == 0
