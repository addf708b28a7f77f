"""p4q_select_noalloc (the selector on the library's per-device scratch
array, for callers that cannot allocate) against p4q_select with a
caller-supplied workspace: the same indices and the same pruned rows, bit for
bit, on two calls in a row whose second input is smaller than the first, plus
the oracle on one sample of each.  Requests larger than the scratch array are
refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from paper_2609_34867_amd import P4QError
from workload import random_features
from gpu_util import Guarded, bits, check_canaries, first_mismatch, to_gpu, to_np

pytestmark = pytest.mark.gpu


def inputs(seed, B, N, d, J, T):
    vis = np.stack([random_features(seed * 10 + b, N, d) for b in range(B)])
    con = np.stack([random_features(seed * 10 + 5 + b, J, d, outliers=0) for b in range(B)])
    txt = np.stack([random_features(seed * 10 + 7 + b, T, d, outliers=0) for b in range(B)])
    return vis, con, txt


def test_noalloc_matches_select_on_two_calls():
    # the second call is smaller than the first in every dimension, so stale
    # scratch contents of the first call lie past what the second one reads
    for seed, (B, N, d, J, T, K) in ((1, (8, 2880, 4096, 4, 64, 640)), (2, (2, 576, 2048, 3, 32, 64))):
        vis, con, txt = inputs(seed, B, N, d, J, T)
        vt, ct, tt = to_gpu(vis), to_gpu(con), to_gpu(txt)
        ref_idx, ref_tok = p4q.select(vt, ct, tt, K)
        gi, gt = Guarded((B, K), torch.int32, "idx_out"), Guarded((B, K + T, d), torch.float16, "tokens_out")
        idx, tok = p4q.select_noalloc(vt, ct, tt, K, idx_out=gi.t, tokens_out=gt.t)
        torch.cuda.synchronize()
        check_canaries(gi, gt)
        assert (m := first_mismatch(to_np(idx), to_np(ref_idx))) is None, (seed, m)
        assert (m := first_mismatch(bits(to_np(tok)), bits(to_np(ref_tok)))) is None, (seed, m)
        ridx, rtok, _, _ = oracle.select(vis[B - 1], con[B - 1], txt[B - 1], K)
        assert np.array_equal(to_np(idx)[B - 1], ridx)
        assert np.array_equal(bits(to_np(tok)[B - 1]), bits(rtok))


def test_noalloc_refuses_requests_beyond_the_scratch():
    # 64 x 2880 tokens with 8 concepts need ~18 MB of workspace (> 8 MiB)
    B, N, d, J, T, K = 64, 2880, 64, 8, 0, 16
    assert p4q.lib().p4q_select_workspace_bytes(B, N, d, J) > 8 << 20
    vt = torch.zeros((B, N, d), dtype=torch.float16, device="cuda")
    ct = torch.zeros((B, J, d), dtype=torch.float16, device="cuda")
    idx = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(P4QError, match="scratch"):
        p4q.select_noalloc(vt, ct, None, K, idx_out=idx)
    torch.cuda.synchronize()
    assert bool((idx == -7).all()), "a refused call wrote its output"
