"""The MLP scorer's entry point that allocates nothing (its scratch is a
library-held device buffer) against the workspace entry point, through the
C ABI: same kernels, same order of sums, so the scores and the kept ids are
bit-identical; two calls in a row, the second smaller than the first (the
buffer keeps the first call's contents), and a size beyond the buffer is
refused before anything is launched."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2608_08020_amd import gambit
from workload.generate import to_bf16_bits

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _bf16(a):
    return torch.from_numpy(to_bf16_bits(np.asarray(a, np.float32)).view(np.int16)).view(torch.bfloat16).to(DEV)


def _case(rng, n, dim, hidden):
    h = _bf16(rng.standard_normal((n, dim)))
    w1 = _bf16(rng.standard_normal((hidden, dim)) / np.sqrt(dim))
    b1 = torch.from_numpy((0.01 * rng.standard_normal(hidden)).astype(np.float32)).to(DEV)
    w2 = torch.from_numpy((rng.standard_normal(hidden) / np.sqrt(hidden)).astype(np.float32)).to(DEV)
    ids = torch.from_numpy(rng.permutation(3 * n)[:n].astype(np.int32)).to(DEV)
    return h, w1, b1, w2, ids


def test_static_scratch_entry_matches_workspace_entry():
    rng = np.random.default_rng(77)
    for n, dim, hidden, act, keep in [(512, 4096, 1024, "relu", 128), (77, 256, 128, "gelu", 9)]:
        h, w1, b1, w2, ids = _case(rng, n, dim, hidden)
        ref_s, ref_k = gambit.mlp_score(h, w1, b1, w2, 0.25, act, ids=ids, keep=keep)
        scores = torch.full((n,), float("nan"), dtype=torch.float32, device=DEV)
        kept = torch.full((keep,), -7, dtype=torch.int32, device=DEV)
        got_s, got_k = gambit.mlp_score_static(h, w1, b1, w2, 0.25, act, ids=ids, keep=keep, scores_out=scores,
                                               keep_out=kept)
        torch.cuda.synchronize()
        assert torch.equal(got_s.view(torch.int32), ref_s.view(torch.int32)), (n, "scores differ")
        assert got_k.cpu().tolist() == ref_k.cpu().tolist(), (n, "kept ids differ")
        # without the ranking
        s2, k2 = gambit.mlp_score_static(h, w1, b1, w2, 0.25, act)
        assert k2 is None and torch.equal(s2.view(torch.int32), ref_s.view(torch.int32))


def test_static_scratch_entry_refuses_sizes_beyond_its_buffer():
    L = gambit.lib()
    n, dim, hidden = 4096, 128, 131136         # 4 * 4096 * ceil(131136 / 128) bytes > 16 MiB
    assert L.gambit_mlp_workspace_size(n, hidden) > gambit.MLP_STATIC_SCRATCH_BYTES
    fake = ctypes.c_void_p(1 << 20)            # never dereferenced: the call fails its size check
    m = gambit.Mlp(dim, hidden, gambit.ACT_RELU, fake.value, fake.value, fake.value, 0.0)
    st = L.gambit_mlp_score_static(n, fake, ctypes.byref(m), fake, None, 0, None, None)
    assert st == gambit.ERR_WORKSPACE
    assert L.gambit_mlp_workspace_size(4096, 131072) <= gambit.MLP_STATIC_SCRATCH_BYTES
