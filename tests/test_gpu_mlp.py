"""GPU parity of the fused 2-layer MLP scorer against the oracle (fp64):
scores within 1e-4 (the probe bar), the fused top-k bit-exact where the
oracle's scores decide it by at least 1e-5; error paths; and the scorer
feeding the tournament's running means (gambit_record_scores) gives the
oracle's tournament."""
import numpy as np
import pytest
import torch

from _tournament import same_ranking
from oracle.formats import bf16_to_f64
from oracle.mlp import mlp_scores
from oracle.pool import PoolModel
from oracle.probe import rank
from oracle.tournament import TournamentModel
from paper_2608_08020_amd import gambit
from paper_2608_08020_amd.gambit import GambitError, Pool, mlp_score
from workload.mlp import MLP_256_32B, MLP_512, MLP_SMALL, MlpConfig, hidden_states, weights

pytestmark = pytest.mark.gpu


def _dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _run(cfg, keep=0):
    W1, b1, w2, b2 = weights(cfg)
    h = hidden_states(cfg)
    ids = torch.arange(cfg.n, dtype=torch.int32, device="cuda")
    got, top = mlp_score(_dev_bf16(h), _dev_bf16(W1), torch.from_numpy(b1).cuda(), torch.from_numpy(w2).cuda(), b2,
                         cfg.act, ids=ids, keep=keep)
    want = mlp_scores(bf16_to_f64(h), bf16_to_f64(W1), b1.astype(np.float64), w2.astype(np.float64), b2, cfg.act)
    return got.cpu().numpy().astype(np.float64), want, (top.cpu().numpy().tolist() if top is not None else None)


@pytest.mark.parametrize("cfg", [MLP_SMALL, MLP_256_32B, MLP_512], ids=lambda c: c.name)
def test_scores_match_oracle(cfg):
    got, want, top = _run(cfg, keep=cfg.n)
    assert np.abs(got - want).max() <= 1e-4
    assert same_ranking(top, rank(range(cfg.n), want), list(want))


def test_top_k_exact_at_the_keep_boundary():
    cfg = MLP_512
    got, want, top = _run(cfg, keep=128)
    order = rank(range(cfg.n), want)
    assert want[order[127]] - want[order[128]] >= 1e-5
    assert top == order[:128]


@pytest.mark.parametrize("n,dim,hidden,act", [(1, 128, 64, "relu"), (17, 384, 192, "gelu"), (64, 640, 64, "relu")])
def test_edge_shapes(n, dim, hidden, act):
    cfg = MlpConfig(name="edge", seed=40 + n, n=n, dim=dim, hidden=hidden, act=act)
    got, want, _ = _run(cfg)
    assert np.abs(got - want).max() <= 1e-4


def test_invalid_shapes_are_rejected():
    for dim, hidden in [(100, 64), (256, 96)]:
        h = torch.zeros((4, dim), dtype=torch.bfloat16, device="cuda")
        w1 = torch.zeros((hidden, dim), dtype=torch.bfloat16, device="cuda")
        b = torch.zeros(hidden, dtype=torch.float32, device="cuda")
        with pytest.raises(GambitError):
            mlp_score(h, w1, b, b, 0.0)
    assert gambit.lib().gambit_mlp_workspace_size(4, 96) == 0


def test_mlp_scores_drive_the_tournament():
    cfg = MlpConfig(name="mlp_tournament", seed=50, n=12, dim=256, hidden=128, act="gelu")
    W1, b1, w2, b2 = weights(cfg)
    p = Pool(num_blocks=256, num_q_heads=4, num_kv_heads=1, max_traces=16, max_blocks_per_trace=8)
    om = TournamentModel(PoolModel(num_blocks=256, n_kv_heads=1, head_dim=128, kv_dtype="bf16", max_traces=16,
                                   max_blocks_per_trace=8))
    ids = list(range(12))
    lens = [10 + 7 * i for i in ids]
    p.kv_alloc(ids, lens)
    om.pool.alloc(ids, lens)
    for rnd in range(3):
        running = om.scheduler_view()
        h = hidden_states(MlpConfig(name="r", seed=60 + rnd, n=len(running), dim=256, hidden=128, act="gelu"))
        f, _ = mlp_score(_dev_bf16(h), _dev_bf16(W1), torch.from_numpy(b1).cuda(), torch.from_numpy(w2).cuda(), b2,
                         "gelu")
        p.record_scores(running, f)
        om.score_update(running, mlp_scores(bf16_to_f64(h), bf16_to_f64(W1), b1.astype(np.float64),
                                            w2.astype(np.float64), b2, "gelu"))
        case, n, pruned, pairs, _ = p.tournament(14, 3, 0)
        res = om.tournament(14, 3, 0)
        assert (case, n, pruned, pairs) == (res.case, res.n_active, res.pruned, res.pairs)
    sb, ns, _, _ = p.trace_state(list(range(16)))
    assert np.abs(sb - np.array(om.sbar)).max() <= 1e-5 and ns.tolist() == om.nsc
    p.pool_check()


def test_exact_ties_rank_by_id():
    """Many hidden states repeated exactly (bit-equal scores) under shuffled,
    non-contiguous ids: the fused ranking is the total order (score
    descending, id ascending) of the scores it returned, and the scores match
    the oracle."""
    cfg = MlpConfig(name="ties", seed=71, n=300, dim=512, hidden=256, act="relu")
    W1, b1, w2, b2 = weights(cfg)
    rng = np.random.default_rng(5)
    src = rng.integers(0, 40, size=cfg.n)
    h = hidden_states(cfg)[src]
    ids = rng.permutation(1000)[:cfg.n].astype(np.int32)
    got, top = mlp_score(_dev_bf16(h), _dev_bf16(W1), torch.from_numpy(b1).cuda(), torch.from_numpy(w2).cuda(), b2,
                         cfg.act, ids=torch.from_numpy(ids).cuda(), keep=cfg.n)
    s = got.cpu().numpy()
    for k in np.unique(src):
        assert np.all(s[src == k] == s[src == k][0]), "copies of one state scored differently"
    order = sorted(range(cfg.n), key=lambda i: (-float(s[i]), int(ids[i])))
    assert top.cpu().numpy().tolist() == [int(ids[i]) for i in order]
    want = mlp_scores(bf16_to_f64(h), bf16_to_f64(W1), b1.astype(np.float64), w2.astype(np.float64), b2, cfg.act)
    assert np.abs(s.astype(np.float64) - want).max() <= 1e-4
