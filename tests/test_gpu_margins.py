"""GPU parity: cure_margins (Sec. 3.3 Eq. 2 and the UFP gate) against the oracle."""

import numpy as np
import pytest
import torch

import oracle
import paper_2608_00531_amd as pc
from synth import preset, make_workload, bf16_round
from parity_util import say, upload, gpu_margins, check_margins, to_dev, MARGIN_TOL

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny_fp32", "llama3_8b_ctx2k_b1"])
def test_preset_margins(name):
    say("margins", name)
    w = preset(name)
    dev = upload(w)
    got = gpu_margins(w, dev)
    torch.cuda.synchronize()
    check_margins(w, got)
    # The planted UFP positions are the lowest-margin chain rows.
    for b in range(w.batch):
        cnt = int(got["ufp_cnt"][b])
        assert sorted(got["ufp_pos"][b, :cnt].tolist()) == w.ufp_planted[b]
        assert np.array_equal(got["top1_idx"][b].cpu().numpy(), w.tgt_planted[b])


def test_ragged_batch16_full_size():
    say("margins llama3_8b_ragged_b16 (768 x 128256 bf16)")
    w = preset("llama3_8b_ragged_b16")
    dev = upload(w)
    got = gpu_margins(w, dev)
    torch.cuda.synchronize()
    check_margins(w, got)


def _rows(vals, dtype):
    x = np.asarray(vals, np.float32)
    return (bf16_round(x) if dtype == "bf16" else x)


def _run_raw(x, dtype, chain_len=0, tau=float("inf"), budget=0, depth=1, gate=False):
    t = to_dev(x, dtype)
    return pc.cure_margins(t, chain_len=chain_len, tau=tau, repair_budget=budget,
                           branch_depth=depth, gate=gate)


def _compare(x, dtype, got):
    ref = oracle.margins(x.reshape(-1, x.shape[-1]), dtype)
    g = {k: v.reshape(-1).cpu().numpy() for k, v in got.items() if k in ref}
    for key in ("top1_idx", "top2_idx", "top1_val", "top2_val"):
        assert np.array_equal(g[key], ref[key]), key
    assert np.array_equal(g["margin"], ref["margin_f32"], equal_nan=True)
    fin = np.isfinite(ref["lse"])
    assert np.array_equal(np.isfinite(g["lse"]), fin)
    assert np.all(np.abs(g["lse"][fin] - ref["lse"][fin]) <= MARGIN_TOL)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_edge_rows(dtype):
    say("margins edge rows", dtype)
    rows = [
        [1.0, 2.0],                              # vocab 2
        [2.0, 2.0],                              # tie at the top: indices 0, 1, margin 0
        [-np.inf, 5.0],
        [-np.inf, -np.inf],                      # all -inf
    ]
    for r in rows:
        x = _rows([r], dtype)[None]
        _compare(x, dtype, _run_raw(x, dtype))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("vocab", [3, 7, 8, 9, 255, 2049, 8193, 40001, 128256, 262147])
def test_random_rows_many_vocab_sizes(dtype, vocab):
    say("margins random rows vocab", vocab, dtype)
    rng = np.random.default_rng(vocab)
    x = (rng.standard_normal((3, 5, vocab)) * 3).astype(np.float32)
    x = _rows(x, dtype)
    _compare(x, dtype, _run_raw(x, dtype))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ties_across_chunks_go_to_lowest_index(dtype):
    say("margins ties across chunks", dtype)
    vocab = 128256
    x = np.zeros((4, vocab), np.float32)
    x[0, [100000, 5, 70000]] = 9.0               # max three times: top1 5, top2 70000
    x[1, [127999, 64001]] = 9.0                  # max twice, far apart
    x[2, 3] = 9.0
    x[2, [128255, 40000]] = 8.5                  # unique max, tie for second
    x[3, :] = -np.inf
    x[3, [77777, 1]] = 1.0
    x = _rows(x, dtype)[None]
    got = _run_raw(x, dtype)
    _compare(x, dtype, got)
    assert got["top1_idx"][0].tolist() == [5, 64001, 3, 1]
    assert got["top2_idx"][0].tolist() == [70000, 127999, 40000, 77777]


def _placement_rows(vocab, rng):
    """Eight rows whose top entries sit where the kernel's wave-wide merges of
    the lanes' best vectors must get them right. Entry 8 v + j is entry j of
    16-byte vector v; with the row in one chunk, vectors v, v + 256 and v + 512
    belong to the same lane, vectors 0-63 to wave 0 and 64-127 to wave 1."""
    E = lambda v, j: 8 * v + j
    r = rng.uniform(-4.0, 4.0, size=(8, vocab)).astype(np.float32)
    r[0, [E(5, 3), E(261, 6), E(517, 0)]] = [20.0, 19.0, 18.0]   # one lane's vectors
    r[1, [E(7, 1), E(7, 6), E(300, 2)]] = [20.0, 19.5, 19.0]     # runner-up in the best vector
    r[2, [E(300, 2), E(40, 7)]] = 20.0                           # equal maxima in two lanes
    r[3, [E(200, 1), E(70, 5), E(130, 0)]] = 20.0                # and across waves
    r[4, [E(9, 0), E(9, 4), E(3, 7)]] = [20.0, 19.0, 19.0]       # runner-up tie across vectors
    r[5, :] = 1.0                                                # constant row
    r[6, :] = -np.inf
    r[6, E(100, 3)] = 0.5                                        # one finite entry
    r[7, [vocab - 1, vocab - 9]] = [20.0, 19.75]                 # the row's last vectors
    return r


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("vocab", [65536, 128256])
@pytest.mark.parametrize("nrows", [8, 520])
def test_top2_vector_placements(dtype, vocab, nrows):
    """Top-2 exactness when the two best vectors share a lane, the runner-up is in
    the best vector, or equal maxima sit in several lanes and waves (the lowest
    index wins). 520 rows keep each row in one chunk; 8 rows split each row."""
    say("margins top-2 placements", dtype, vocab, nrows)
    rng = np.random.default_rng(vocab + nrows)
    special = _rows(_placement_rows(vocab, rng), dtype)
    x = np.empty((nrows, vocab), special.dtype)       # bf16: raw bits
    x[:8] = special
    if nrows > 8:
        x[8:] = _rows(rng.uniform(-4.0, 4.0, size=(nrows - 8, vocab)), dtype)
    got = _run_raw(x[None], dtype)
    ref = oracle.margins(special, dtype)
    g = {k: v.reshape(-1)[:8].cpu().numpy() for k, v in got.items() if k in ref}
    for key in ("top1_idx", "top2_idx", "top1_val", "top2_val"):
        assert np.array_equal(g[key], ref[key]), key
    assert np.array_equal(g["margin"], ref["margin_f32"], equal_nan=True)
    fin = np.isfinite(ref["lse"])
    assert np.array_equal(np.isfinite(g["lse"]), fin)
    assert np.all(np.abs(g["lse"][fin] - ref["lse"][fin]) <= MARGIN_TOL)
    E = lambda v, j: 8 * v + j
    assert g["top1_idx"].tolist()[:6] == [E(5, 3), E(7, 1), E(40, 7), E(70, 5), E(9, 0), 0]
    assert g["top2_idx"].tolist()[:6] == [E(261, 6), E(7, 6), E(300, 2), E(130, 0), E(3, 7), 1]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unaligned_row_stride_uses_scalar_path(dtype):
    say("margins unaligned ld", dtype)
    rng = np.random.default_rng(9)
    full = (rng.standard_normal((6, 5003)) * 2).astype(np.float32)
    full = _rows(full, dtype)
    t = to_dev(full, dtype)[:, 1:5001]           # row stride 5003, first row offset by 1
    got = pc.cure_margins(t.unsqueeze(0).squeeze(0), gate=False)
    _compare(full[:, 1:5001][None], dtype, got)


def test_large_values_and_negative_rows():
    say("margins large/negative values")
    rng = np.random.default_rng(4)
    x = (rng.standard_normal((2, 4, 30000)) * 3).astype(np.float32)
    x[0] += 1000.0
    x[1] -= 1000.0
    _compare(x, "f32", _run_raw(x, "f32"))


def test_ufp_gate_variants():
    say("margins UFP gate variants")
    w = make_workload("g", batch=3, hq=4, hkv=1, d=64, vocab=5000, ctx_lens=[8, 8, 8],
                      chain_len=16, n_ufp=5, branch_depth=2, seed=41)
    dev = upload(w)
    for tau, budget, depth in [(1.0, 10, 2), (0.3, 10, 2), (np.inf, 100, 1), (1.0, 3, 4),
                               (-np.inf, 8, 1), (0.7, 7, 3)]:
        got = pc.cure_margins(dev["logits"], chain_len=w.chain_len, tau=float(tau),
                              repair_budget=budget, branch_depth=depth)
        for b in range(w.batch):
            ref = oracle.margins(w.logits[b], "bf16")
            want = oracle.ufp_select(ref["margin_f32"][: w.chain_len], tau, budget, depth)
            cnt = int(got["ufp_cnt"][b])
            assert got["ufp_pos"][b, :cnt].tolist() == want, (tau, budget, depth)
            assert all(p == -1 for p in got["ufp_pos"][b, cnt:].tolist())
    # chain_len == rows
    got = pc.cure_margins(dev["logits"], chain_len=w.n_max, tau=1.0, repair_budget=64,
                          branch_depth=1)
    for b in range(w.batch):
        ref = oracle.margins(w.logits[b], "bf16")
        want = oracle.ufp_select(ref["margin_f32"], 1.0, 64, 1)
        assert got["ufp_pos"][b, : int(got["ufp_cnt"][b])].tolist() == want


def test_repeated_calls_reuse_workspace():
    say("margins repeated calls")
    w = preset("llama3_8b_ctx2k_b1")
    dev = upload(w)
    first = gpu_margins(w, dev)
    for _ in range(5):
        again = gpu_margins(w, dev)
    torch.cuda.synchronize()
    for k in first:
        assert torch.equal(first[k], again[k]), k


def test_workspace_reuse_across_shapes():
    # One cached workspace serves calls of different shapes in any order.
    say("margins workspace reuse across shapes")
    rng = np.random.default_rng(12)
    shapes = [(2, 40, 60000), (1, 3, 9000), (4, 16, 128256), (1, 2, 17), (3, 7, 33333)]
    for batch, rows, vocab in shapes + shapes[::-1]:
        x = _rows((rng.standard_normal((batch, rows, vocab)) * 3).astype(np.float32), "bf16")
        got = _run_raw(x, "bf16", chain_len=rows, tau=1.0, budget=rows, depth=1, gate=True)
        _compare(x, "bf16", got)
        for b in range(batch):
            ref = oracle.margins(x[b], "bf16")
            want = oracle.ufp_select(ref["margin_f32"], 1.0, rows, 1)
            assert got["ufp_pos"][b, : int(got["ufp_cnt"][b])].tolist() == want


@pytest.mark.parametrize("seed", range(16))
def test_random_shapes_strides_and_gate(seed):
    # Seeded random batches: row count, vocabulary (2 .. 300000, log-uniform),
    # dtype, a row stride past the vocabulary (odd strides take the scalar
    # path), ties at the top, rows with many -inf entries, and the UFP gate
    # with random tau, budget and branch depth.
    rng = np.random.default_rng(5000 + seed)
    batch = int(rng.integers(1, 5))
    rows = int(rng.integers(1, 40))
    vocab = int(np.exp(rng.uniform(np.log(2), np.log(300000))))
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    pad = int(rng.choice([0, 0, 1, 3, 8]))
    say("margins random", seed, batch, rows, vocab, dtype, pad)
    x = (rng.standard_normal((batch, rows, vocab + pad)) * rng.uniform(0.5, 6)).astype(np.float32)
    for b in range(batch):
        for r in range(rows):
            u = rng.random()
            if u < 0.2:
                j = rng.integers(0, vocab, size=int(rng.integers(2, 5)))
                x[b, r, j] = x[b, r, :vocab].max() + 1.0
            elif u < 0.3:
                x[b, r, rng.integers(0, vocab, size=max(1, vocab // 3))] = -np.inf
    x = _rows(x, dtype)
    chain = int(rng.integers(1, rows + 1))
    tau = float(rng.choice([np.inf, 1.0, 0.3, 2.5]))
    depth = int(rng.integers(1, 6))
    budget = int(rng.integers(0, 4 * chain + 1))
    t = to_dev(x, dtype)[:, :, :vocab]
    got = pc.cure_margins(t, chain_len=chain, tau=tau, repair_budget=budget, branch_depth=depth)
    torch.cuda.synchronize()
    _compare(np.ascontiguousarray(x[:, :, :vocab]), dtype,
             {k: v for k, v in got.items() if k not in ("ufp_pos", "ufp_cnt")})
    for b in range(batch):
        ref = oracle.margins(x[b, :, :vocab], dtype)
        want = oracle.ufp_select(ref["margin_f32"][:chain], tau, budget, depth)
        cnt = int(got["ufp_cnt"][b])
        assert got["ufp_pos"][b, :cnt].tolist() == want
        assert all(p == -1 for p in got["ufp_pos"][b, cnt:].tolist())
