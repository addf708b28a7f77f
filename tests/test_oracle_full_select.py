"""Pins for the oracle's three-stage selector (O3': Sec. 3.2, Eq.
p4q_progressive_selection -- Query Relevance, Visual Saliency over the tokens
left, Visual Diversity completion).

Each check is independent of the oracle's own loops: exact rational budget
arithmetic, numpy lexsort for the saliency ranking, a hand-derived worked
example for the max-min greedy, and float64 cosines of the dequantized
copies recomputed from scratch at every greedy step.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from workload import CONFIGS, cls_attention, random_features, selector_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "diversity_worked_example.txt")


def test_stage_budgets_exact_floor():
    """floor(0.3 K), floor(0.2 K), remainder -- in exact rationals, never in
    binary floating point (192 * 0.3 = 57.599999... in float64)."""
    assert oracle.stage_budgets(640) == (192, 128, 320)
    assert oracle.stage_budgets(320) == (96, 64, 160)
    assert oracle.stage_budgets(192) == (57, 38, 97)
    assert oracle.stage_budgets(64) == (19, 12, 33)
    assert oracle.stage_budgets(1) == (0, 0, 1)
    for K in range(1, 3000):
        kq, ks, kd = oracle.stage_budgets(K)
        assert kq == int(Fraction(3, 10) * K) and ks == int(Fraction(2, 10) * K)
        assert kq + ks + kd == K and kd >= 0


def test_saliency_matches_lexsort_with_ties():
    rng = np.random.default_rng(5)
    a = rng.random(300).astype(np.float32)
    a[[10, 40, 41, 200]] = a[7]                          # planted ties
    a[[3, 4]] = np.float32(0.0)
    kept = [1, 7, 99, 250]
    rem = np.array([i for i in range(300) if i not in kept])
    order = rem[np.lexsort((rem, -a[rem].astype(np.float64)))]
    for k in (0, 1, 5, 37, len(rem)):
        assert oracle.saliency_topk(a, kept, k) == [int(i) for i in order[:k]]


def _golden():
    rows, meta = [], {}
    for line in open(GOLDEN):
        line = line.split("#", 1)[0].split()
        if not line:
            continue
        if line[0].startswith("x"):
            rows.append([float(v) for v in line[1:]])
        else:
            meta[line[0]] = [int(v) for v in line[1:]]
    return np.array(rows, dtype=np.float16), meta


def test_diversity_worked_example():
    x, meta = _golden()
    cv, s = oracle.quantize_rows(x)
    assert np.array_equal(cv, x.astype(np.int64)) and s[0] == 1.0
    picks = oracle.diversity_greedy(cv, meta["kept"], len(meta["picks"]),
                                    np.zeros(len(x), np.float32))
    assert picks == meta["picks"]


def _float_maxcos(vf, S, cand):
    """max cosine to S of every candidate, float64, from the dequantized rows."""
    n = np.linalg.norm(vf, axis=1)
    out = {}
    for i in cand:
        best = -np.inf
        for t in S:
            c = 0.0 if n[i] == 0 or n[t] == 0 else float(vf[i] @ vf[t]) / (n[i] * n[t])
            best = max(best, c)
        out[i] = best
    return out


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_diversity_greedy_is_maxmin_in_float64(seed):
    """At every step the oracle's pick minimizes the max cosine to the current
    retained set, recomputed from scratch in float64 from the dequantized
    vectors; a lower-index candidate is never strictly (by 1e-12) better."""
    x = random_features(seed, 48, 64, outliers=2, scale=4.0)
    cv, sc = oracle.quantize_rows(x)
    vf = oracle.dequantize_rows(cv, sc).astype(np.float64)
    kept = [0, 5, 9]
    picks = oracle.diversity_greedy(cv, kept, 20, np.zeros(48, np.float32))
    S = list(kept)
    for p in picks:
        cand = [i for i in range(48) if i not in S]
        m = _float_maxcos(vf, S, cand)
        lo = min(m.values())
        assert m[p] <= lo + 1e-12
        assert not any(m[i] < m[p] - 1e-12 for i in cand if i < p)
        S.append(p)
    assert len(set(picks)) == len(picks) and not set(picks) & set(kept)


def test_diversity_duplicates_last_and_opposites_first():
    """A copy of a retained token (cos 1) goes last; its negation (cos -1)
    goes first."""
    x = random_features(11, 16, 32).astype(np.float32)
    x[3] = x[0]          # duplicate of the retained token 0
    x[12] = -x[0]        # its opposite
    x = x.astype(np.float16)
    cv, _ = oracle.quantize_rows(x)
    picks = oracle.diversity_greedy(cv, [0], 15, np.zeros(16, np.float32))
    assert picks[0] == 12 and picks[-1] == 3


def test_diversity_empty_retained_set_seeds_with_saliency():
    x = random_features(12, 20, 32)
    a = np.linspace(0.1, 0.9, 20).astype(np.float32)
    a[7] = 5.0
    cv, _ = oracle.quantize_rows(x)
    assert oracle.diversity_greedy(cv, [], 3, a)[0] == 7


def test_full_selector_properties():
    cfg = CONFIGS["tiny"]
    si = selector_inputs(cfg, samples=[0])
    a = cls_attention(cfg.cfg_id, cfg.N, 0)
    K = cfg.K
    kq, ks, kd = oracle.stage_budgets(K)
    idx, tok, (qp, sp, dp) = oracle.select_full(si.vis[0], si.concepts[0], a, si.text[0], K, kq, ks)
    assert len(idx) == K and np.all(np.diff(idx) > 0)
    assert (len(qp), len(sp), len(dp)) == (kq, ks, kd)
    cv, _ = oracle.quantize_rows(si.vis[0])
    cq, _ = oracle.quantize_rows(si.concepts[0])
    assert qp == [int(i) for i in oracle.select_query_relevance(cv, cq, kq)]
    rest = [i for i in range(cfg.N) if i not in qp]
    assert sp == sorted(rest, key=lambda i: (-float(a[i]), i))[:ks]
    assert set(qp) | set(sp) | set(dp) == set(int(i) for i in idx)
    assert np.array_equal(tok[:K].view(np.uint16), si.vis[0][idx].view(np.uint16))
    assert np.array_equal(tok[K:].view(np.uint16), si.text[0].view(np.uint16))


def test_full_selector_reduces_to_query_relevance():
    """alpha = 1 (kq = K): the hot-path selector."""
    cfg = CONFIGS["tiny"]
    si = selector_inputs(cfg, samples=[0])
    a = cls_attention(cfg.cfg_id, cfg.N, 0)
    idx, tok, _ = oracle.select_full(si.vis[0], si.concepts[0], a, si.text[0], cfg.K, cfg.K, 0)
    ridx, rtok, _, _ = oracle.select(si.vis[0], si.concepts[0], si.text[0], cfg.K)
    assert np.array_equal(idx, ridx)


def test_full_selector_scale_invariant():
    """Scaling the features by 2 leaves every code, hence the selection, alone."""
    x = random_features(21, 96, 64)
    con = random_features(22, 3, 64)
    a = cls_attention(9, 96, 0)
    t = random_features(23, 4, 64)
    i1, _, _ = oracle.select_full(x, con, a, t, 24, 7, 4)
    i2, _, _ = oracle.select_full((x.astype(np.float32) * 2).astype(np.float16), con, a, t, 24, 7, 4)
    assert np.array_equal(i1, i2)
