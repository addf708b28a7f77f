"""GPU parity of p4q_w4a4_linear against the oracle: int32 accumulators and
fp16/bf16 outputs must match bit for bit (the epilogue's operation order is
fixed, so 'within 1e-3 relative' is met with zero error)."""
import functools

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34867_amd as p4q
from workload import CONFIGS, random_features, weight, attn_standin
from gpu_util import Guarded, bits, check_canaries, first_mismatch, to_gpu, to_np

pytestmark = pytest.mark.gpu


def codes_for(M, N, K, seed, extreme=None):
    rng = np.random.default_rng(seed)
    if extreme is None:
        a = rng.integers(-8, 8, size=(M, K)).astype(np.int8)
        w = rng.integers(-8, 8, size=(N, K)).astype(np.int8)
    else:
        a = np.full((M, K), extreme, dtype=np.int8)
        w = np.full((N, K), extreme, dtype=np.int8)
    sa = rng.uniform(1e-3, 4, size=M).astype(np.float32)
    sw = rng.uniform(1e-4, 3e-2, size=N).astype(np.float32)
    return oracle.pack_int4(a), sa, oracle.pack_int4(w), sw


def run_gpu(ap, sa, wp, sw, out_dtype, with_acc=True, workspace=None):
    """One call into canary-guarded outputs; with_acc=False runs the y-only
    kernels (the instantiations the benchmark times)."""
    tdt = torch.float16 if out_dtype == "fp16" else torch.bfloat16
    M, N = ap.shape[0], wp.shape[0]
    gy = Guarded((M, N), tdt, "y")
    ga = Guarded((M, N), torch.int32, "acc_out") if with_acc else None
    p4q.w4a4_linear(to_gpu(ap), to_gpu(sa), to_gpu(wp), to_gpu(sw), y=gy.t,
                    acc_out=None if ga is None else ga.t, workspace=workspace)
    torch.cuda.synchronize()
    check_canaries(gy, *([ga] if ga else []))
    return to_np(gy.t), (to_np(ga.t) if ga else None)


def check_full(ap, sa, wp, sw, out_dtype):
    """Both instantiations (with and without the int32 store) against the
    oracle, bit for bit."""
    racc, ry = oracle.w4a4_linear(ap, sa, wp, sw, out_dtype)
    y, acc = run_gpu(ap, sa, wp, sw, out_dtype)
    assert (m := first_mismatch(acc, racc.astype(np.int32))) is None, m
    assert (m := first_mismatch(bits(y), bits(ry))) is None, m
    y, _ = run_gpu(ap, sa, wp, sw, out_dtype, with_acc=False)
    assert (m := first_mismatch(bits(y), bits(ry))) is None, ("y-only", m)


@pytest.mark.parametrize("out_dtype", ["fp16", "bf16"])
@pytest.mark.parametrize("shape", [(1, 1, 32), (5, 17, 96), (16, 16, 128), (130, 250, 288),
                                   (127, 129, 4096), (256, 384, 1024), (1, 4096, 4096),
                                   (4, 300, 11008), (300, 64, 13824), (257, 129, 5120)])
def test_shapes(shape, out_dtype):
    M, N, K = shape
    check_full(*codes_for(M, N, K, M * 7 + N), out_dtype)


@pytest.mark.parametrize("shape", [(1030, 1100, 512), (1024, 1024, 4128), (1500, 2100, 96),
                                   (2304, 1280, 11008), (1024, 4096, 32)])
def test_large_tile_shapes(shape):
    """Shapes served by the 256 x 128 two-blocks-per-CU kernel, with ragged
    M, N and K tails."""
    M, N, K = shape
    check_full(*codes_for(M, N, K, M + N + K), "bf16")


@pytest.mark.parametrize("shape", [(17, 1024, 32), (130, 1100, 288), (517, 1030, 4128),
                                   (1000, 2100, 96), (300, 1024, 8224), (45, 1040, 6016)])
def test_mid_tile_shapes(shape):
    """Shapes served by the 128 x 128 tiles of the same kernel (16 < M <
    1024, N >= 1024), ragged in M, N and K: unsplit (no workspace) and, where
    the shape has few tiles, with K split across work-groups (the last
    slice holding the ragged k-tile), each with and without the int32
    store."""
    M, N, K = shape
    ap, sa, wp, sw = codes_for(M, N, K, M + 3 * N + K)
    check_full(ap, sa, wp, sw, "fp16")
    nws = p4q.lib().p4q_w4a4_linear_workspace_bytes(M, N, K)
    if nws:
        racc, ry = oracle.w4a4_linear(ap, sa, wp, sw, "bf16")
        ws = p4q.w4a4_linear_workspace(M, N, K, torch.device("cuda:0"))
        for with_acc in (True, False):
            y, acc = run_gpu(ap, sa, wp, sw, "bf16", with_acc=with_acc, workspace=ws)
            if with_acc:
                assert (m := first_mismatch(acc, racc.astype(np.int32))) is None, m
            assert (m := first_mismatch(bits(y), bits(ry))) is None, (with_acc, m)


@pytest.mark.parametrize("extreme", [-8, 7])
def test_extreme_codes_large_K(extreme):
    """|acc| = 64 * K at K = 65536 (and 49 K with +7): checks the int32 range of
    the scaled MFMA accumulation."""
    check_full(*codes_for(40, 36, 65536, 3, extreme), "bf16")
    check_full(*codes_for(1040, 1030, 65536, 3, extreme), "fp16")


def test_strided_output():
    ap, sa, wp, sw = codes_for(33, 40, 256, 9)
    y = torch.full((33, 48), -1.0, dtype=torch.bfloat16, device="cuda")
    p4q.w4a4_linear(to_gpu(ap), to_gpu(sa), to_gpu(wp), to_gpu(sw), y=y[:, :wp.shape[0]])
    torch.cuda.synchronize()
    _, ry = oracle.w4a4_linear(ap, sa, wp, sw, "bf16")
    got = to_np(y)
    assert np.array_equal(bits(got[:, :40]), bits(ry))
    assert np.all(bits(got[:, 40:]) == 0xBF80)           # -1.0 untouched


def test_quantized_pipeline_tiny():
    """quant_act -> w4a4_linear on the tiny config's real recipe (fp16 out)."""
    cfg = CONFIGS["tiny"]
    x = random_features(5, cfg.M, 4096)
    w = weight(cfg, 0)
    xq = p4q.quant_act(to_gpu(x))
    wq = p4q.quant_act(to_gpu(w))
    y, acc = p4q.w4a4_linear(*xq, *wq, torch.float16, return_acc=True)
    torch.cuda.synchronize()
    ap, sa = oracle.quant_act(x)
    wp, sw = oracle.quant_act(w)
    racc, ry = oracle.w4a4_linear(ap, sa, wp, sw, "fp16")
    assert np.array_equal(to_np(acc), racc.astype(np.int32))
    assert np.array_equal(bits(to_np(y)), bits(ry))


def check_sampled(ap, sa, wp, sw, y, acc, rng, edge_rows=32, entries=1024):
    """First and last rows in full plus random entries, against the oracle
    (acc may be None: the y-only kernels)."""
    M = ap.shape[0]
    for rows in (slice(0, edge_rows), slice(M - edge_rows, M)):
        racc, ry = oracle.w4a4_linear(ap[rows], sa[rows], wp, sw, "bf16")
        if acc is not None:
            assert (m := first_mismatch(acc[rows], racc.astype(np.int32))) is None, m
        assert (m := first_mismatch(bits(y[rows]), bits(ry))) is None, m
    yb = bits(y)
    for _ in range(entries):
        m, n = int(rng.integers(M)), int(rng.integers(wp.shape[0]))
        racc, ry = oracle.w4a4_linear_entry(ap, sa, wp, sw, m, n, "bf16")
        assert yb[m, n] == ry, (m, n)
        if acc is not None:
            assert acc[m, n] == racc, (m, n)


def launch_weights(cfg, members):
    """Row-concatenated quantized weights of one launch of the layer, from the
    config's weight recipe (quantized by the oracle)."""
    parts = [oracle.quant_act(weight(cfg, li)) for li in members]
    return np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts])


@pytest.mark.slow
@pytest.mark.parametrize("members", [(0, 1, 2), (3,), (4, 5), (6,)],
                         ids=["qkv", "o_proj", "gate_up", "down_proj"])
def test_llava_next_b16_launches_sampled(members):
    """The four launches one benchmark step times at M = 11264 (q|k|v 12288 x
    4096 and gate|up 22016 x 4096 on row-concatenated weights, o_proj 4096 x
    4096, down_proj 4096 x 11008), in the y-only instantiation the benchmark
    runs and in the one that also stores the int32 accumulators; the first and
    last 32 rows and 1024 random entries of each are checked against the
    oracle."""
    cfg = CONFIGS["next7b_b16"]
    k_in = cfg.linears[members[0]].k_in
    rng = np.random.default_rng(sum(members) + 17 * len(members))
    ap = rng.integers(0, 256, size=(cfg.M, k_in // 2), dtype=np.uint8)
    sa = rng.uniform(1e-3, 4, size=cfg.M).astype(np.float32)
    wp, sw = launch_weights(cfg, members)
    y, _ = run_gpu(ap, sa, wp, sw, "bf16", with_acc=False)
    check_sampled(ap, sa, wp, sw, y, None, rng)
    y2, acc = run_gpu(ap, sa, wp, sw, "bf16")
    assert np.array_equal(bits(y), bits(y2)), "y differs between the two instantiations"
    check_sampled(ap, sa, wp, sw, y2, acc, rng, entries=256)


@pytest.mark.slow
@pytest.mark.parametrize("NK", [(15360, 5120), (5120, 5120), (27648, 5120), (5120, 13824)],
                         ids=["qkv", "o_proj", "gate_up", "down_proj"])
def test_stress13b_prefill_launches_sampled(NK):
    """The 13B-shape prefill launches at M = 5632 (batch 8 x (640 + 64)):
    h = 5120, f = 13824, random codes and scales, y-only (the timed kernel)
    and with the accumulators, sampled against the oracle."""
    N, K = NK
    M = CONFIGS["stress13b_b8"].M
    rng = np.random.default_rng(N + K)
    ap = rng.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    wp = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    sa = rng.uniform(1e-3, 4, size=M).astype(np.float32)
    sw = rng.uniform(1e-4, 3e-2, size=N).astype(np.float32)
    y, _ = run_gpu(ap, sa, wp, sw, "bf16", with_acc=False)
    check_sampled(ap, sa, wp, sw, y, None, rng, entries=512)
    y2, acc = run_gpu(ap, sa, wp, sw, "bf16")
    assert np.array_equal(bits(y), bits(y2))
    check_sampled(ap, sa, wp, sw, y2, acc, rng, edge_rows=16, entries=256)


@pytest.mark.parametrize("M", [1, 2, 4, 7, 16])
@pytest.mark.parametrize("NK", [(5120, 5120), (5120, 13824), (1000, 4128), (33, 32), (47, 224),
                                (200, 6176), (200, 8224), (72, 14336)])
def test_decode_gemv_shapes(M, NK):
    """M <= 16 runs the HBM-streaming decode kernel: ragged N (not a multiple
    of its 16-row groups), K not a multiple of its 128-value k-tiles, K split
    unevenly over its wavefronts (8 up to K = 6144, 16 beyond: 6176 and 8224
    are the first rows past a launch-shape boundary, 14336 the longest row),
    every M in the padded 16-row operand."""
    N, K = NK
    check_full(*codes_for(M, N, K, 31 * M + N + K), "bf16" if M % 2 else "fp16")


@pytest.mark.parametrize("extreme", [-8, 7])
def test_decode_gemv_extreme_codes(extreme):
    check_full(*codes_for(16, 40, 65536, 5, extreme), "bf16")


def test_decode_gemv_strided_output():
    ap, sa, wp, sw = codes_for(3, 70, 512, 13)
    y = torch.full((3, 80), -1.0, dtype=torch.bfloat16, device="cuda")
    p4q.w4a4_linear(to_gpu(ap), to_gpu(sa), to_gpu(wp), to_gpu(sw), y=y[:, :wp.shape[0]])
    torch.cuda.synchronize()
    _, ry = oracle.w4a4_linear(ap, sa, wp, sw, "bf16")
    got = to_np(y)
    assert np.array_equal(bits(got[:, :70]), bits(ry))
    assert np.all(bits(got[:, 70:]) == 0xBF80)


@functools.lru_cache(maxsize=None)
def _weights_13b(li):
    cfg = CONFIGS["stress13b_b8"]
    w = weight(cfg, li)
    return (w,) + tuple(oracle.quant_act(w))


@pytest.mark.slow
@pytest.mark.parametrize("M", [1, 4, 16])
def test_decode_13b_layer(M):
    """Decode step of the 13B-shape stress config: quantized decode-step
    activations against all seven quantized linears (weights from the
    config's recipe), bit-exact."""
    from workload import gemv_activations
    cfg = CONFIGS["stress13b_b8"]
    for li, lin in enumerate(cfg.linears):
        w, wp, sw = _weights_13b(li)
        x = gemv_activations(cfg, M, lin.k_in)
        xq = p4q.quant_act(to_gpu(x))
        wq = p4q.quant_act(to_gpu(w))
        y, acc = p4q.w4a4_linear(*xq, *wq, torch.bfloat16, return_acc=True)
        torch.cuda.synchronize()
        ap, sa = oracle.quant_act(x)
        racc, ry = oracle.w4a4_linear(ap, sa, wp, sw, "bf16")
        assert (m := first_mismatch(to_np(acc), racc.astype(np.int32))) is None, (lin.name, m)
        assert (m := first_mismatch(bits(to_np(y)), bits(ry))) is None, (lin.name, m)


def test_decode_graph_replay_matches_eager():
    """The decode linears captured in a HIP graph (as a serving loop runs
    them): every replay, with eager work and synchronizations in between,
    reproduces the eager outputs bit for bit."""
    shapes = [(5120, 5120), (13824, 5120), (5120, 13824)]
    M = 4
    ops = [codes_for(M, N, K, 100 + i) for i, (N, K) in enumerate(shapes)]
    ins = [tuple(to_gpu(x) for x in op) for op in ops]
    ref = [p4q.w4a4_linear(*args, torch.bfloat16) for args in ins]
    ys = [torch.empty_like(r) for r in ref]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for args, yv in zip(ins, ys):
            p4q.w4a4_linear(*args, y=yv)
    for rep in range(3):
        for yv in ys:
            yv.fill_(float(rep + 1))                      # eager work between replays
        junk = p4q.w4a4_linear(*ins[rep % 3], torch.bfloat16)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for r, yv in zip(ref, ys):
            assert torch.equal(r.view(torch.int16), yv.view(torch.int16)), rep
        del junk


@pytest.mark.parametrize("shape,split", [((384, 4096, 11008), True), ((256, 4096, 4096), True),
                                         ((96, 512, 4096), True), ((704, 4096, 11008), True),
                                         ((384, 4096, 4096), True), ((704, 4096, 4096), True),
                                         ((384, 12288, 4096), True), ((520, 8200, 2080), True),
                                         ((300, 8200, 4096), True), ((512, 16384, 4096), False)])
def test_small_m_split_k(shape, split):
    """Batch-1 shapes (one image's pruned sequence).  Given the workspace,
    the tiles past the last whole round per CU (all of them when there are
    fewer tiles than CUs) are split along K across work-groups that meet in
    the workspace; (K_in <= 4096) 64-row tiles fill the CUs where 128-row
    tiles are too few; 512 tiles of 128 x 128 divide evenly and run
    unsplit.  (520, 8200, 2080): ragged in M, N and the last k-tile, with
    512 whole tiles of 64 rows and 73 split in three; (300, 8200, 4096) the
    same with a ragged last 64-row tile.  Every path must equal the oracle
    bit for bit, in bf16 and in fp16."""
    M, N, K = shape
    assert (p4q.lib().p4q_w4a4_linear_workspace_bytes(M, N, K) > 0) == split
    ap, sa, wp, sw = codes_for(M, N, K, seed=M + N)
    racc, ry = oracle.w4a4_linear(ap, sa, wp, sw, "bf16")
    dev = torch.device("cuda:0")
    empty = torch.empty(0, dtype=torch.uint8, device=dev)      # zero bytes: the unsplit path
    shared = p4q.w4a4_linear_workspace(M, N, K, dev)
    for ws in (None, empty):
        for with_acc in (True, False, True):  # the split epilogue with and without acc_out
            y, acc = run_gpu(ap, sa, wp, sw, "bf16", with_acc=with_acc,
                             workspace=ws if ws is not None else shared)
            if with_acc:
                assert (m := first_mismatch(acc, racc.astype(np.int32))) is None, m
            assert (m := first_mismatch(bits(y), bits(ry))) is None, (with_acc, m)
            if ws is None and shared is not None and N >= 1024:
                # the tile kernel's arrival counters are back at zero for the
                # next call (the small-M kernel's slices have no counters)
                assert int(shared[:4096].count_nonzero()) == 0
    if shared is not None:                    # the fp16-output instances of the split path
        _, ry16 = oracle.w4a4_linear(ap, sa, wp, sw, "fp16")
        for with_acc in (False, True):
            y, acc = run_gpu(ap, sa, wp, sw, "fp16", with_acc=with_acc, workspace=shared)
            if with_acc:
                assert (m := first_mismatch(acc, racc.astype(np.int32))) is None, m
            assert (m := first_mismatch(bits(y), bits(ry16))) is None, ("fp16", with_acc, m)


@pytest.mark.parametrize("cfg_name", ["next7b_b1_k320", "next7b_b1_k640", "llava15_7b"])
def test_batch1_layer_launches(cfg_name):
    """The four launches of a batch-1 decoder layer (M = 384 / 704 / 256) as
    the benchmark runs them (y only, split-K workspace given), in full against
    the oracle on random codes."""
    cfg = CONFIGS[cfg_name]
    dev = torch.device("cuda:0")
    h, f = cfg.d, cfg.linears[4].n_out
    for N, K in ((3 * h, h), (h, h), (2 * f, h), (h, f)):
        ap, sa, wp, sw = codes_for(cfg.M, N, K, seed=N + K + cfg.M)
        racc, ry = oracle.w4a4_linear(ap, sa, wp, sw, "bf16")
        y, _ = run_gpu(ap, sa, wp, sw, "bf16", with_acc=False,
                       workspace=p4q.w4a4_linear_workspace(cfg.M, N, K, dev))
        assert (m := first_mismatch(bits(y), bits(ry))) is None, ((N, K), m)


@pytest.mark.parametrize("shape", [(384, 12288, 4096), (384, 4096, 11008)])
def test_split_k_graph_replays(shape):
    """The in-launch split (remainder tiles, and a launch whose tiles are all
    split) under HIP graph capture: its arrival counters are reset by the
    kernel itself, with no memset node, so every replay must reproduce the
    oracle's y, also with eager calls on the same workspace between replays."""
    M, N, K = shape
    dev = torch.device("cuda:0")
    ap, sa, wp, sw = codes_for(M, N, K, seed=7 * M + N)
    _, ry = oracle.w4a4_linear(ap, sa, wp, sw, "bf16")
    ws = p4q.w4a4_linear_workspace(M, N, K, dev)
    assert ws is not None
    a, s_a, w, s_w = to_gpu(ap), to_gpu(sa), to_gpu(wp), to_gpu(sw)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    p4q.w4a4_linear(a, s_a, w, s_w, y=y, workspace=ws)     # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        p4q.w4a4_linear(a, s_a, w, s_w, y=y, workspace=ws)
    for rep in range(3):
        y.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        assert (m := first_mismatch(bits(to_np(y)), bits(ry))) is None, (rep, m)
        assert int(ws[:4096].count_nonzero()) == 0, rep
        y2 = torch.empty_like(y)
        p4q.w4a4_linear(a, s_a, w, s_w, y=y2, workspace=ws)   # eager call between replays
        torch.cuda.synchronize()
        assert (m := first_mismatch(bits(to_np(y2)), bits(ry))) is None, (rep, m)
    del g
