"""GPU parity of p4q_select against the oracle: per-token integer statistics
(D, Nv), retained indices and the gathered sequence must match bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import CONFIGS, selector_inputs, random_features
from gpu_util import Guarded, bits, check_canaries, first_mismatch, to_gpu, to_np

pytestmark = pytest.mark.gpu


def run_gpu(vis, con, text, K, dtype, clip=1.0, ws=None, reps=3):
    """`reps` calls on one workspace (filled with garbage first unless given):
    nothing of an earlier call may leak into a later one, and rows are
    claimed dynamically, so every call must give the same outputs bit for
    bit; the last one's are returned."""
    B, N, d = vis.shape
    J = con.shape[1]
    vt, ct = to_gpu(vis, dtype), to_gpu(con, dtype)
    tt = None if text is None else to_gpu(text, dtype)
    T = 0 if text is None else text.shape[1]
    if ws is None:
        ws = p4q.select_workspace(B, N, d, J, vt.device)
        ws.fill_(0xA5)
    outs = []
    for _ in range(reps):
        gi = Guarded((B, K), torch.int32, "idx_out")
        gt = Guarded((B, K + T, d), vt.dtype, "tokens_out")
        idx, tok = p4q.select(vt, ct, tt, K, clip, idx_out=gi.t, tokens_out=gt.t, workspace=ws)
        torch.cuda.synchronize()
        check_canaries(gi, gt)
        stats = to_np(ws[: B * N * (J + 1) * 4].view(torch.int32)).reshape(B, N, J + 1)
        outs.append((to_np(idx), to_np(tok), stats))
    for r in range(1, reps):
        for a, b_, what in zip(outs[0], outs[r], ("idx", "tokens", "stats")):
            assert np.array_equal(bits(a) if a.dtype.kind == "f" else a,
                                  bits(b_) if b_.dtype.kind == "f" else b_), f"call {r} {what} differs"
    return outs[-1]


def check(vis, con, text, K, dtype="fp16", clip=1.0, samples=None, ws=None):
    B = vis.shape[0]
    T = 0 if text is None else text.shape[1]
    idx, tok, stats = run_gpu(vis, con, text, K, dtype, clip, ws=ws)
    for b in (range(B) if samples is None else samples):
        tb = text[b] if T else np.zeros((0, vis.shape[2]), dtype=vis.dtype)
        ridx, rtok, D, Nv = oracle.select(vis[b], con[b], tb, K, dtype, clip)
        assert (m := first_mismatch(stats[b, :, :-1], D.astype(np.int32))) is None, f"D b={b}: {m}"
        assert (m := first_mismatch(stats[b, :, -1], Nv.astype(np.int32))) is None, f"Nv b={b}: {m}"
        assert (m := first_mismatch(idx[b], ridx)) is None, f"idx b={b}: {m}"
        assert (m := first_mismatch(bits(tok[b]), bits(rtok))) is None, f"tokens b={b}: {m}"


def synth(seed, B, N, d, J, T, dtype="fp16", dup=False):
    vis = np.stack([random_features(seed * 10 + b, N, d, dtype) for b in range(B)])
    con = np.stack([random_features(seed * 10 + 5 + b, J, d, dtype, outliers=0)
                    for b in range(B)])
    text = None if T == 0 else np.stack([random_features(seed * 10 + 7 + b, T, d, dtype,
                                                         outliers=0) for b in range(B)])
    if dup:                      # duplicate rows -> exact score ties across indices
        for b in range(B):
            vis[b, 5::7] = vis[b, 3]
            vis[b, 6::11] = vis[b, 9]
    return vis, con, text


def test_tiny_config():
    cfg = CONFIGS["tiny"]
    si = selector_inputs(cfg)
    check(si.vis, si.concepts, si.text, cfg.K)


@pytest.mark.parametrize("J", [1, 2, 3, 4, 7, 8])
def test_concept_counts(J):
    vis, con, text = synth(J, 2, 300, 512, J, 8)
    check(vis, con, text, 41)


@pytest.mark.parametrize("K", [1, 2, 3, 64, 299, 300])
def test_budget_edges(K):
    vis, con, text = synth(11, 1, 300, 256, 4, 5)
    check(vis, con, text, K)


def test_ties_and_ragged_N():
    vis, con, text = synth(12, 3, 1000, 1024, 4, 16, dup=True)
    check(vis, con, text, 97)


def test_no_text_bf16_and_clip():
    vis, con, _ = synth(13, 2, 777, 768, 3, 0, dtype="bf16")
    check(vis, con, None, 100, dtype="bf16")
    check(vis, con, None, 100, dtype="bf16", clip=0.6)


def test_zero_and_identical_rows():
    vis, con, text = synth(14, 1, 200, 256, 3, 4)
    vis[0, 10:20] = 0                      # Nv = 0 -> cosine 0
    con[0, 1] = 0                          # Nq = 0 -> index order for concept 1
    vis[0, 50] = con[0, 0]                 # cosine exactly 1 for concept 0
    vis[0, 51] = -con[0, 2]                # cosine exactly -1 for concept 2
    check(vis, con, text, 60)


def test_max_N_and_wide_d():
    vis, con, text = synth(15, 1, 8192, 128, 2, 2)
    check(vis, con, text, 512)
    vis, con, text = synth(16, 1, 70, 8192, 2, 2)
    check(vis, con, text, 9)


@pytest.mark.parametrize("name", ["next7b_b1_k320", "next7b_b1_k640"])
def test_llava_next_b1(name):
    cfg = CONFIGS[name]
    si = selector_inputs(cfg)
    check(si.vis, si.concepts, si.text, cfg.K)


@pytest.mark.slow
def test_llava_next_b16_sampled():
    """The batch-16 LLaVA-NeXT workload in one launch (as the benchmark runs
    it); samples 0, 7 and 15 are checked against the oracle in full, and every
    sample's indices are checked for being sorted, distinct and in range."""
    cfg = CONFIGS["next7b_b16"]
    si = selector_inputs(cfg)
    check(si.vis, si.concepts, si.text, cfg.K, samples=[0, 7, 15])
    idx, _, _ = run_gpu(si.vis, si.concepts, si.text, cfg.K, "fp16")
    for b in range(cfg.B):
        assert np.all(np.diff(idx[b]) > 0) and idx[b][0] >= 0 and idx[b][-1] < cfg.N


@pytest.mark.slow
def test_13b_shape_sampled():
    cfg = CONFIGS["stress13b_b8"]
    si = selector_inputs(cfg, samples=[0, 5])
    check(si.vis, si.concepts, si.text, cfg.K)


def test_workspace_reused_for_another_shape():
    """One workspace buffer for three shapes in turn (B*N kept, so the
    internal offsets coincide): every call must match the oracle."""
    d, J = 256, 3
    ws = p4q.select_workspace(2, 300, d, J, torch.device("cuda:0"))
    ws.fill_(0x5A)
    v1, c1, t1 = synth(41, 1, 600, d, J, 4)
    check(v1, c1, t1, 50, ws=ws)
    v2, c2, t2 = synth(42, 2, 300, d, J, 4)
    check(v2, c2, t2, 40, ws=ws)
    v3, c3, t3 = synth(43, 1, 600, d, J, 4)
    check(v3, c3, t3, 64, ws=ws)
