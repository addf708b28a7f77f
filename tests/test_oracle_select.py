"""Pins for the oracle's quantization-aware Query-Relevance selector (O3).

The selector ranks visual tokens, per query concept, by the cosine similarity
of fake-quantized copies (Sec. 3.2, Eq. p4q_progressive_selection and the
Query Relevance paragraph).  The checks below are independent of the oracle's
sort-and-walk: Cauchy-Schwarz, self-similarity, float64 cosines of the
dequantized copies, and brute-force ranks from pairwise exact comparisons.
"""
import itertools

import numpy as np
import pytest

import oracle
from workload import random_features, CONFIGS, selector_inputs


def _precedes(Di, Nvi, Dk, Nvk, i, k):
    """Exact 'token i ranks before token k' by integer cross-multiplication.
    Scores are D/sqrt(Nv*Nq); Nq > 0 is common to both and cancels."""
    def sgn(v):
        return (v > 0) - (v < 0)
    if Nvi == 0 and Nvk == 0:
        return i < k
    if Nvi == 0:          # score_i = 0
        return 0 > sgn(Dk) or (Dk == 0 and i < k)
    if Nvk == 0:
        return sgn(Di) > 0 or (Di == 0 and i < k)
    li = sgn(Di) * Di * Di * Nvk
    lk = sgn(Dk) * Dk * Dk * Nvi
    return li > lk or (li == lk and i < k)


def brute_force_select(cv, cq, K):
    """Stage-wise selection from pairwise ranks (O(N^2) per concept)."""
    D = [[int(sum(int(a) * int(b) for a, b in zip(v, q))) for q in cq] for v in cv]
    Nv = [int(sum(int(a) * int(a) for a in v)) for v in cv]
    Nq = [int(sum(int(a) * int(a) for a in q)) for q in cq]
    N, J = len(cv), len(cq)
    quotas = [K // J + (1 if j < K % J else 0) for j in range(J)]
    S = set()
    for j in range(J):
        cand = [i for i in range(N) if i not in S]
        for i in cand:
            if Nq[j] == 0:
                rank = sum(1 for k in cand if k < i)
            else:
                rank = sum(1 for k in cand if k != i and
                           _precedes(D[k][j], Nv[k], D[i][j], Nv[i], k, i))
            if rank < quotas[j]:
                S.add(i)
    return sorted(S)


def _tiny_inputs(seed, N, d, J, levels):
    rng = np.random.default_rng(seed)
    vis = rng.integers(-levels, levels + 1, size=(N, d)).astype(np.float16)
    con = rng.integers(-levels, levels + 1, size=(J, d)).astype(np.float16)
    return vis, con


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("J", [1, 2, 3])
def test_brute_force_tiny(seed, J):
    N, d = 11, 8
    vis, con = _tiny_inputs(seed, N, d, J, levels=2 if seed % 2 else 7)
    if seed % 3 == 0:                    # duplicated rows -> exact score ties
        vis[5] = vis[2]
        vis[9] = vis[2]
    cv, _ = oracle.quantize_rows(vis)
    cq, _ = oracle.quantize_rows(con)
    for K in range(1, N + 1):
        got = oracle.select_query_relevance(cv, cq, K).tolist()
        assert got == brute_force_select(cv, cq, K), (K, J)


def test_subset_enumeration_J1():
    """J = 1: the kept set is the unique K-subset whose members all rank
    before every dropped token."""
    vis, con = _tiny_inputs(101, 9, 6, 1, 3)
    vis[4] = vis[1]
    cv, _ = oracle.quantize_rows(vis)
    cq, _ = oracle.quantize_rows(con)
    D, Nv, Nq = oracle.concept_dots(cv, cq)
    for K in range(1, 10):
        winners = []
        for S in itertools.combinations(range(9), K):
            rest = [k for k in range(9) if k not in S]
            if all(_precedes(int(D[i, 0]), int(Nv[i]), int(D[k, 0]), int(Nv[k]), i, k)
                   for i in S for k in rest):
                winners.append(list(S))
        assert len(winners) == 1
        assert oracle.select_query_relevance(cv, cq, K).tolist() == winners[0]


def test_cosine_equals_dequantized_fp64():
    """The integer-code cosine equals CosSim of the real fake-quantized copies
    s*code (scales cancel); a wrong sign or a dropped term shows here."""
    vis = random_features(21, 50, 96)
    con = random_features(22, 3, 96, outliers=0)
    cv, sv = oracle.quantize_rows(vis)
    cq, sq = oracle.quantize_rows(con)
    D, Nv, Nq = oracle.concept_dots(cv, cq)
    vq = oracle.dequantize_rows(cv, sv)
    qq = oracle.dequantize_rows(cq, sq)
    cos64 = (vq @ qq.T) / np.outer(np.linalg.norm(vq, axis=1), np.linalg.norm(qq, axis=1))
    cos_int = D / np.sqrt(np.outer(Nv, Nq).astype(np.float64))
    assert np.allclose(cos64, cos_int, rtol=0, atol=1e-12)
    for i in range(50):
        for j in range(3):
            c2 = float(oracle.signed_cos2(D[i, j], Nv[i], Nq[j]))
            assert abs(c2 - cos64[i, j] * abs(cos64[i, j])) < 1e-12


def test_cauchy_schwarz_and_self_similarity():
    vis = random_features(23, 64, 128)
    con = np.concatenate([vis[10:11], -vis[20:21], random_features(24, 2, 128)])
    cv, _ = oracle.quantize_rows(vis)
    cq, _ = oracle.quantize_rows(con)
    D, Nv, Nq = oracle.concept_dots(cv, cq)
    assert np.all(D.astype(object) ** 2 <= np.outer(Nv, Nq).astype(object))
    assert oracle.signed_cos2(D[10, 0], Nv[10], Nq[0]) == 1
    assert oracle.signed_cos2(D[20, 1], Nv[20], Nq[1]) == -1
    # the identical token ranks first for its concept
    assert oracle.concept_order(D, Nv, Nq, 0)[0] == 10


def test_J1_matches_argsort_of_float_cosines():
    """J = 1 reduces to a plain top-K of the cosine; compare with a stable
    float64 argsort where no two distinct cosines are closer than 1e-9."""
    vis = random_features(25, 300, 256)
    con = random_features(26, 1, 256, outliers=0)
    cv, sv = oracle.quantize_rows(vis)
    cq, sq = oracle.quantize_rows(con)
    vq, qq = oracle.dequantize_rows(cv, sv), oracle.dequantize_rows(cq, sq)
    cos = (vq @ qq[0]) / (np.linalg.norm(vq, axis=1) * np.linalg.norm(qq[0]))
    order = np.lexsort((np.arange(300), -np.round(cos, 12)))
    for K in (1, 17, 64, 150, 300):
        assert oracle.select_query_relevance(cv, cq, K).tolist() == sorted(order[:K].tolist())


def test_concept_permutation_invariance_J1_and_quotas():
    assert oracle.concept_quotas(64, 4) == [16, 16, 16, 16]
    assert oracle.concept_quotas(10, 4) == [3, 3, 2, 2]
    assert oracle.concept_quotas(3, 4) == [1, 1, 1, 0]
    assert sum(oracle.concept_quotas(641, 7)) == 641


def test_zero_concept_orders_by_index():
    vis = random_features(27, 20, 32)
    con = np.zeros((1, 32), dtype=np.float16)
    cv, _ = oracle.quantize_rows(vis)
    cq, _ = oracle.quantize_rows(con)
    assert oracle.select_query_relevance(cv, cq, 5).tolist() == [0, 1, 2, 3, 4]


def test_select_forwards_original_rows():
    cfg = CONFIGS["tiny"]
    si = selector_inputs(cfg)
    idx, tok, D, Nv = oracle.select(si.vis[0][:96], si.concepts[0], si.text[0], 16)
    assert idx.tolist() == sorted(idx.tolist()) and len(set(idx.tolist())) == 16
    assert np.array_equal(tok[:16].view(np.uint16), si.vis[0][idx].view(np.uint16))
    assert np.array_equal(tok[16:].view(np.uint16), si.text[0].view(np.uint16))


def test_fake_quant_changes_selection():
    """On the outlier distribution, selecting from fake-quantized copies differs
    from selecting on the raw features (the quantization awareness is live)."""
    cfg = CONFIGS["tiny"]
    si = selector_inputs(cfg)
    vis, con = si.vis[0], si.concepts[0]
    idx_q = oracle.select_query_relevance(*[oracle.quantize_rows(a)[0] for a in (vis, con)], 64)
    vf, cf = vis.astype(np.float64), con.astype(np.float64)
    cos = (vf @ cf.T) / np.outer(np.linalg.norm(vf, axis=1), np.linalg.norm(cf, axis=1))
    kept = []
    for j, quota in enumerate(oracle.concept_quotas(64, 4)):
        order = np.lexsort((np.arange(vf.shape[0]), -cos[:, j]))
        kept += [int(i) for i in order if i not in kept][:quota]
    repl = 1 - len(set(kept) & set(idx_q.tolist())) / 64
    assert repl > 0.1
