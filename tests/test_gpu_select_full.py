"""GPU parity of p4q_select_full (the three-stage selector of Sec. 3.2)
against the oracle: the Query-Relevance set, the Visual-Saliency set, the
Visual-Diversity picks in pick order, the final ascending indices and the
gathered sequence must all match exactly."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import CONFIGS, cls_attention, random_features, selector_inputs
from gpu_util import Guarded, bits, check_canaries, first_mismatch, to_gpu, to_np

pytestmark = pytest.mark.gpu


def run_gpu(vis, con, cls, text, K, kq, ks, dtype, clip=1.0):
    B, N, d = vis.shape
    vt, ct = to_gpu(vis, dtype), to_gpu(con, dtype)
    at = torch.from_numpy(np.ascontiguousarray(cls, dtype=np.float32)).cuda()
    tt = None if text is None else to_gpu(text, dtype)
    T = 0 if text is None else text.shape[1]
    gi, gs = Guarded((B, K), torch.int32, "idx_out"), Guarded((B, K), torch.int32, "stages_out")
    gt = Guarded((B, K + T, d), vt.dtype, "tokens_out")
    idx, tok, stages = p4q.select_full(vt, ct, at, tt, K, kq, ks, clip, idx_out=gi.t,
                                       stages_out=gs.t, tokens_out=gt.t, return_stages=True)
    torch.cuda.synchronize()
    check_canaries(gi, gs, gt)
    return to_np(idx), to_np(tok), to_np(stages)


def check(vis, con, cls, text, K, kq, ks, dtype="fp16", clip=1.0, samples=None):
    B = vis.shape[0]
    T = 0 if text is None else text.shape[1]
    idx, tok, stages = run_gpu(vis, con, cls, text, K, kq, ks, dtype, clip)
    for b in (range(B) if samples is None else samples):
        tb = text[b] if T else np.zeros((0, vis.shape[2]), dtype=vis.dtype)
        ridx, rtok, (q, s, dp) = oracle.select_full(vis[b], con[b], cls[b], tb, K, kq, ks,
                                                    dtype, clip)
        ref_stages = np.array(sorted(q) + sorted(s) + list(dp), dtype=np.int32)
        assert (m := first_mismatch(stages[b, :kq], ref_stages[:kq])) is None, f"query b={b}: {m}"
        assert (m := first_mismatch(stages[b, kq:kq + ks], ref_stages[kq:kq + ks])) is None, \
            f"saliency b={b}: {m}"
        assert (m := first_mismatch(stages[b, kq + ks:], ref_stages[kq + ks:])) is None, \
            f"diversity b={b}: {m}"
        assert (m := first_mismatch(idx[b], ridx)) is None, f"idx b={b}: {m}"
        assert (m := first_mismatch(bits(tok[b]), bits(rtok))) is None, f"tokens b={b}: {m}"


def synth(seed, B, N, d, J, T, dtype="fp16", dup=False, zeros=False, cls_ties=False):
    vis = np.stack([random_features(seed * 10 + b, N, d, dtype) for b in range(B)])
    con = np.stack([random_features(seed * 10 + 5 + b, J, d, dtype, outliers=0)
                    for b in range(B)])
    text = None if T == 0 else np.stack([random_features(seed * 10 + 7 + b, T, d, dtype,
                                                         outliers=0) for b in range(B)])
    cls = np.stack([cls_attention(100 + seed, N, b) for b in range(B)])
    if dup:                      # duplicated rows -> exactly equal cosines
        for b in range(B):
            vis[b, 5::7] = vis[b, 3]
            vis[b, 6::11] = vis[b, 9]
    if zeros:                    # all-zero rows -> zero code vectors (cosine 0)
        vis[:, 2::13] = 0
    if cls_ties:
        cls[:, 1::5] = cls[:, :1]
    return vis, con, cls, text


def test_tiny_config_paper_budgets():
    cfg = CONFIGS["tiny"]
    si = selector_inputs(cfg)
    cls = np.stack([cls_attention(cfg.cfg_id, cfg.N, b) for b in range(cfg.B)])
    kq, ks, _ = oracle.stage_budgets(cfg.K)
    check(si.vis, si.concepts, cls, si.text, cfg.K, kq, ks)


@pytest.mark.parametrize("kq,ks", [(0, 0), (0, 20), (20, 0), (30, 30), (100, 0), (0, 100),
                                   (40, 60)])
def test_stage_budget_edges(kq, ks):
    """kq = ks = 0 seeds the diversity stage with the most salient token;
    kd = 0 (kq + ks = K) skips it."""
    vis, con, cls, text = synth(21, 2, 300, 256, 3, 5)
    check(vis, con, cls, text, 100, kq, ks)


@pytest.mark.parametrize("K", [1, 2, 299, 300])
def test_total_budget_edges(K):
    vis, con, cls, text = synth(22, 1, 300, 128, 2, 3)
    kq, ks, _ = oracle.stage_budgets(K)
    check(vis, con, cls, text, K, kq, ks)


def test_ties_zero_rows_and_ragged_N():
    """Duplicated rows (equal cosines), zero code vectors and equal CLS
    weights: every tie resolves to the lower index."""
    vis, con, cls, text = synth(23, 2, 1000, 512, 4, 8, dup=True, zeros=True, cls_ties=True)
    check(vis, con, cls, text, 250, 75, 50)


def test_gram_on_the_large_tile_kernel():
    """N >= 1024 takes the 256 x 128 MFMA kernel for the Gram matrices."""
    vis, con, cls, text = synth(24, 2, 1500, 384, 4, 4)
    check(vis, con, cls, text, 300, 90, 60)


def test_bf16_clip_no_text():
    vis, con, cls, _ = synth(25, 2, 777, 768, 3, 0, dtype="bf16")
    check(vis, con, cls, None, 150, 45, 30, dtype="bf16")
    check(vis, con, cls, None, 150, 45, 30, dtype="bf16", clip=0.6)


def test_max_tokens_per_thread():
    """N = 8192: eight candidates per thread of the greedy work-group."""
    vis, con, cls, text = synth(26, 1, 8192, 64, 2, 2)
    check(vis, con, cls, text, 60, 18, 12)


def test_llava_next_b16_sampled():
    """The full LLaVA-NeXT-7B batch (16 x 2880 x 4096, K = 640 at the paper's
    split 192 / 128 / 320) in one call, checked on the first and last
    samples."""
    cfg = CONFIGS["next7b_b16"]
    si = selector_inputs(cfg)
    cls = np.stack([cls_attention(cfg.cfg_id, cfg.N, b) for b in range(cfg.B)])
    kq, ks, _ = oracle.stage_budgets(cfg.K)
    check(si.vis, si.concepts, cls, si.text, cfg.K, kq, ks, samples=[0, cfg.B - 1])
