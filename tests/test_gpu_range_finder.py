"""End-to-end parity of rrf_run against the oracle.

Bar (per workload): the same k; ||Q^T Q - I||_F <= 1e-12 (f64) / 1e-5 (f32);
||A - Q B||_F / ||A||_F <= 1.05x the oracle's (100 u where both sit at
roundoff); projector distance <= 1e-8 (f64) / 1e-3 (f32) on spectral-gap
inputs.  Small and scaled workloads run the oracle live; the five full-size
workloads compare with the oracle's stored k and residual
(tests/golden/oracle_configs.json, written by tests/golden/make_golden.py)
plus the properties that hold at any size.
"""

import json
import os

import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import (ORTH_TOL, PROJ_TOL, gpu_metrics_torch, orth_err,
                            projector_distance, rel_residual, residual_bound,
                            say, to_dev, to_host)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2608_28941_amd as rrf  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "oracle_configs.json")


def _tdt(dtype):
    return torch.float64 if np.dtype(dtype) == np.float64 else torch.float32


def _run(A, w, k_max=0, stop=rrf.RRF_STOP_TRAILING):
    with rrf.Plan(_tdt(w.dtype), A.shape[0], A.shape[1], w.block_b, k_max) as p:
        p.set_stop_mode(stop)
        Q, B, k = p.run(to_dev(A), w.tol, w.block_b, w.sketch_seed)
        tr = p.trace()
        st = p.last_status
        return to_host(Q), to_host(B), k, tr, st


_ORACLE = {}


def _oracle(w, A, k_max=0, stop="trailing"):
    """The oracle's result for workload w (cached: several GPU variants of the
    same workload compare with one oracle run)."""
    key = (w, k_max, stop)
    if key not in _ORACLE:
        _ORACLE[key] = oracle.hbarrf(A, w.tol, w.block_b, w.sketch_seed, k_max=k_max,
                                     dtype=w.np_dtype, stop=stop)
    return _ORACLE[key]


def _elementwise_bound(A, k, w):
    """Q is unique given Omega (Theorem 3.1 + the sign convention); its
    columns agree with the oracle's to about cond(A Omega_k) u, and B's
    entries to that times ||A||_2."""
    dt = np.dtype(w.dtype)
    Om = oracle.normal_v1(w.sketch_seed, A.shape[1], 0, k, dtype=dt).astype(np.float64)
    sv = np.linalg.svd(A.astype(np.float64) @ Om, compute_uv=False)
    tol = 1e3 * (sv[0] / sv[-1]) * np.finfo(dt).eps
    return tol, tol * np.linalg.norm(A.astype(np.float64), 2)


def _check_against_live_oracle(w, A, gap=False, elementwise=False):
    ref = _oracle(w, A)
    say(f"run {w.name} m={w.m} n={w.n} b={w.block_b} tol={w.tol} oracle k={ref.k}")
    Q, B, k, tr, _ = _run(A, w)
    assert k == ref.k
    dt = np.dtype(w.dtype)
    assert orth_err(Q) <= ORTH_TOL[dt]
    res_o = rel_residual(A, ref.Q, ref.B)
    assert rel_residual(A, Q, B) <= residual_bound(res_o, dt)
    # The per-block stopping quantity follows the oracle's.
    assert tr["nblocks"] == len(ref.trace)
    for (kk, e_t, _), g_t in zip(ref.trace, tr["E_trail"]):
        assert abs(g_t - e_t) <= 1e-3 * max(e_t, 1e-6 * ref.E0) + 1e3 * np.finfo(dt).eps * ref.E0
    if gap and k > 0:
        assert projector_distance(Q, ref.Q) <= PROJ_TOL[dt]
    if elementwise and k > 0:
        tq, tb = _elementwise_bound(A, k, w)
        assert np.max(np.abs(Q - ref.Q)) <= tq
        assert np.max(np.abs(B - ref.B)) <= tb
    return Q, B, k, ref


def test_tiny_config_full_size():
    w = W.WORKLOADS["tiny_fp64_500x300"]
    _check_against_live_oracle(w, W.build_matrix(w), elementwise=True)


SCALED = [
    ("galore_fp32_4096x4096", 1024, 1024, None, None),
    ("mlp_fp32_4096x11008", 512, 1376, None, None),
    ("square_fp64_16384", 2048, 2048, None, 1e-5),
    ("tall_fp64_131072x2048", 8192, 256, None, None),
    ("tiny_fp64_500x300", 333, 250, 24, 1e-5),      # b not a power of two
    ("galore_fp32_4096x4096", 700, 900, 48, 2e-2),  # ragged everywhere
]


@pytest.mark.parametrize("name,m,n,b,tol", SCALED)
def test_scaled_workloads(name, m, n, b, tol):
    # Element by element, in the default configuration: the look-ahead with
    # the Gram panel inside the update's launch (blocks of b > 32 columns of
    # these small matrices run as 32-column sub-blocks).
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    _check_against_live_oracle(w, W.build_matrix(w), elementwise=True)


@pytest.mark.parametrize("name,m,n,b,tol", [SCALED[1], SCALED[2], SCALED[5]])
def test_scaled_workloads_64_column_subblocks(monkeypatch, name, m, n, b, tol):
    # Element by element with 64-column sub-blocks (the width large matrices
    # take, e.g. 16384 x 16384): the column-by-column look-ahead path
    # (update_panel_kernel with its fused sample, the redundant panel update
    # in thin_apply_kernel, block 0's panel beside the first sample).
    monkeypatch.setenv("RRF_SUBBLOCK", "64")
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    _check_against_live_oracle(w, W.build_matrix(w), elementwise=True)


@pytest.mark.parametrize("name,m,n,b,tol", [SCALED[0], SCALED[2], SCALED[3], SCALED[5]])
def test_scaled_workloads_tsqr_panel(monkeypatch, name, m, n, b, tol):
    # Same bar with the tall-skinny QR panel (chosen at plan creation).
    monkeypatch.setenv("RRF_PANEL", "tsqr")
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    _check_against_live_oracle(w, W.build_matrix(w))


@pytest.mark.parametrize("name,m,n,b,tol", [SCALED[0], SCALED[1], SCALED[2], SCALED[3],
                                            SCALED[4], SCALED[5]])
def test_scaled_workloads_without_lookahead(monkeypatch, name, m, n, b, tol):
    # Same bar with the look-ahead off (every panel in its own launch, no
    # redundant panel update, no block-0 sample/panel launch; b <= 32: the
    # Gram panel, queued during the stop test).
    monkeypatch.setenv("RRF_LOOKAHEAD", "0")
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    _check_against_live_oracle(w, W.build_matrix(w), elementwise=True)


@pytest.mark.parametrize("name,m,n,b,tol", SCALED)
def test_scaled_workloads_gram_panel(monkeypatch, name, m, n, b, tol):
    # Same bar with the Gram-matrix panel (chosen at plan creation).
    monkeypatch.setenv("RRF_PANEL", "gram")
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    _check_against_live_oracle(w, W.build_matrix(w))


@pytest.mark.parametrize("name", W.GAP_INPUTS)
def test_gap_inputs_gram_panel(monkeypatch, name):
    monkeypatch.setenv("RRF_PANEL", "gram")
    w = W.WORKLOADS[name]
    _check_against_live_oracle(w, W.build_matrix(w), gap=True)


@pytest.mark.parametrize("name", W.GAP_INPUTS)
def test_gap_inputs(name):
    w = W.WORKLOADS[name]
    A = W.build_matrix(w)
    Q, B, k, ref = _check_against_live_oracle(w, A, gap=True)
    if "exact_rank48" in name:
        assert k == 48
    else:
        assert k == 128


def test_wide_and_tall_and_degenerate():
    for (m, n, b, tol) in [(40, 300, 16, 1e-3), (300, 40, 16, 0.0), (65, 65, 64, 1e-9),
                           (1, 50, 1, 0.5), (50, 1, 4, 1e-6)]:
        w = W.Workload(f"edge{m}x{n}", m, n, "float64", b, tol, 5, 6,
                       kind="lowrank_noise", rank=min(m, n), noise=1e-3,
                       spectrum="pow10_i_over_30")
        _check_against_live_oracle(w, W.build_matrix(w))
    # A = 0 and tol >= 1 give k = 0.
    with rrf.Plan(torch.float64, 30, 20, 8) as p:
        Q, B, k = p.run(to_dev(np.zeros((30, 20))), 1e-3, 8, 1)
        assert k == 0 and Q.shape == (30, 0) and B.shape == (0, 20)
        A = W.random_dense(30, 20, np.float64, 3)
        assert p.run(to_dev(A), 1.0, 8, 1)[2] == 0


def test_rank_cap_warns_and_tolerance_zero_runs_to_cap():
    w = W.scaled("tiny_fp64_500x300", 200, 120, block_b=16, tol=1e-9)
    A = W.build_matrix(w)
    Q, B, k, _, st = _run(A, w, k_max=40)
    assert k == 40 and st == rrf.RRF_WARN_KMAX
    ref = oracle.hbarrf(A, w.tol, 16, w.sketch_seed, k_max=40)
    assert projector_distance(Q, ref.Q) < 1e-10
    w0 = W.scaled("tiny_fp64_500x300", 200, 120, block_b=16, tol=0.0)
    Q, B, k, tr, st = _run(A, w0)
    assert k == 120 and st == rrf.RRF_OK
    assert orth_err(Q) <= 1e-12


def test_subtract_mode_matches_oracle():
    w = W.scaled("square_fp64_16384", 1024, 800, block_b=32, tol=1e-4)
    A = W.build_matrix(w)
    ref = oracle.hbarrf(A, w.tol, w.block_b, w.sketch_seed, stop="subtract")
    Q, B, k, tr, _ = _run(A, w, stop=rrf.RRF_STOP_SUBTRACT)
    assert k == ref.k
    for (_, _, e_s), g in zip(ref.trace, tr["E_sub"]):
        assert abs(g - e_s) <= 1e-9 * ref.E0


@pytest.mark.parametrize("lookahead", ["1", "0"])
def test_lookahead_tall_panel_elementwise(monkeypatch, lookahead):
    # 12288 rows at b = 64: the panel inside the look-ahead launch holds 64
    # rows per thread (panels above 8192 rows); k = 320 in five blocks,
    # E / sigma^2 = 3.0 at k = 256 and 0.17 at 320.
    monkeypatch.setenv("RRF_LOOKAHEAD", lookahead)
    monkeypatch.setenv("RRF_SUBBLOCK", "64")
    w = W.scaled("square_fp64_16384", 12288, 384, block_b=64, tol=1e-2)
    _, _, k, _ = _check_against_live_oracle(w, W.build_matrix(w), elementwise=True)
    assert k == 320


@pytest.mark.parametrize("name,m,n,b,tol,wgs", [
    ("galore_fp32_4096x4096", 1024, 1024, 32, None, 64),   # 4 rows per thread, 32 workgroups
    ("galore_fp32_4096x4096", 1024, 1024, 32, None, 16),   # 8 rows per thread
    ("galore_fp32_4096x4096", 1024, 1024, 32, None, 8),    # 16 rows per thread
    ("tall_fp64_131072x2048", 8192, 256, None, None, 64),  # 16 rows per thread, 64 workgroups
    ("tiny_fp64_500x300", 500, 300, 16, 1e-4, 64),         # 16 columns, 4 rows per thread
    ("tiny_fp64_500x300", 500, 300, 16, 1e-4, 4),          # 8 rows per thread
    ("tiny_fp64_500x300", 500, 300, 16, 1e-4, 2),          # 16 rows per thread
    ("tiny_fp64_500x300", 333, 250, 20, 1e-5, 64),         # 20 of 32 columns, ragged
])
def test_lookahead_gram_panel_shapes(monkeypatch, name, m, n, b, tol, wgs):
    # Blocks of at most 32 columns: the next block's Gram panel runs on the
    # first workgroups of the update's launch; RRF_LA_GRAM_WGS caps its grid,
    # which picks the rows per thread.  Element by element against the
    # oracle.
    monkeypatch.setenv("RRF_LA_GRAM_WGS", str(wgs))
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    _check_against_live_oracle(w, W.build_matrix(w), elementwise=True)


def test_deterministic_repeat_lookahead_gram():
    # Bit-identical results from two runs of the Gram look-ahead path (b = 32).
    w = W.scaled("tall_fp64_131072x2048", 8192, 256)
    A = to_dev(W.build_matrix(w))
    with rrf.Plan(torch.float64, 8192, 256, 32) as p:
        Q1, B1, k1 = p.run(A, w.tol, 32, w.sketch_seed)
        Q2, B2, k2 = p.run(A, w.tol, 32, w.sketch_seed)
        torch.cuda.synchronize()
        assert k1 == k2 and k1 > 32
        assert torch.equal(Q1, Q2) and torch.equal(B1, B2)


@pytest.mark.parametrize("sub", ["64", "auto"])
@pytest.mark.parametrize("name,m,n,b,tol", [
    ("square_fp64_16384", 2048, 2048, 128, 1e-5),    # two 64-column sub-blocks
    ("tiny_fp64_500x300", 333, 250, 100, 1e-5),      # sub-blocks of 64 and 36
    ("galore_fp32_4096x4096", 1024, 1024, 80, 2e-2), # 64 and 16: mixed panel routes
])
def test_blocks_wider_than_64(monkeypatch, name, m, n, b, tol, sub):
    # block_b > 64 runs as sub-blocks of at most 64 columns (32 for these
    # small matrices by default) with the stop test at block ends; the oracle
    # factors each block whole.
    if sub != "auto":
        monkeypatch.setenv("RRF_SUBBLOCK", sub)
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    _, _, k, ref = _check_against_live_oracle(w, W.build_matrix(w), elementwise=True)
    assert k % b == 0 or k == min(m, n)


def test_panel_beyond_register_capacity():
    # 131072 rows at b = 64: no register-resident panel grid holds the panel,
    # so it takes the tall-skinny QR tree.  Fixed rank k = 128 (tol = 0,
    # k_cap = n); the oracle is the plain definition of the result
    # (Theorem 3.1): the Householder QR of A Omega_k (the oracle's geqr2 and
    # org2r) and B = Q^T A.
    w = W.scaled("tall_fp64_131072x2048", 131072, 128, block_b=64, tol=0.0)
    A = W.build_matrix(w)
    say("tall 131072x128 b=64: oracle plain definition")
    Om = oracle.normal_v1(w.sketch_seed, 128, 0, 128, dtype=np.float64)
    Vo, tauo = oracle.geqr2(A @ Om)
    Qo = oracle.org2r(Vo, tauo)
    Bo = Qo.T @ A
    say("tall 131072x128 b=64: rrf_run")
    Q, B, k, _, st = _run(A, w)
    assert k == 128 and st == rrf.RRF_OK
    tq, tb = _elementwise_bound(A, k, w)
    assert np.max(np.abs(Q - Qo)) <= tq
    assert np.max(np.abs(B - Bo)) <= tb
    assert orth_err(Q) <= ORTH_TOL[np.dtype(np.float64)]


def test_deterministic_repeat_lookahead(monkeypatch):
    # Bit-identical results from two runs of the look-ahead path (b = 64,
    # 64-column sub-blocks).
    monkeypatch.setenv("RRF_SUBBLOCK", "64")
    w = W.scaled("square_fp64_16384", 2048, 2048, tol=1e-5)
    A = to_dev(W.build_matrix(w))
    with rrf.Plan(torch.float64, 2048, 2048, 64) as p:
        Q1, B1, k1 = p.run(A, w.tol, 64, w.sketch_seed)
        Q2, B2, k2 = p.run(A, w.tol, 64, w.sketch_seed)
        torch.cuda.synchronize()
        assert k1 == k2 and k1 > 64
        assert torch.equal(Q1, Q2) and torch.equal(B1, B2)


def test_wait_give_up_is_reported(monkeypatch):
    # A spin limit of 0 (set from the host) makes every grid-wide wait give
    # up at its first poll; each kernel still runs to its end.  The run and
    # the stage entry points must report RRF_ERR_INTERNAL, and a plan with the
    # default limit must work afterwards.
    monkeypatch.setenv("RRF_TEST_SPIN_LIMIT", "0")
    w = W.scaled("square_fp64_16384", 1024, 1024, tol=1e-5)
    A = W.build_matrix(w)
    Ad = to_dev(A)
    say("wait give-up: rrf_run, rrf_panel_qr, thin rrf_apply_block_reflector")
    with rrf.Plan(torch.float64, 1024, 1024, 64) as p:
        with pytest.raises(rrf.RRFError) as e:
            p.run(Ad, w.tol, 64, w.sketch_seed)
        assert e.value.status == -6
        Y = to_dev(W.random_dense(1024, 64, np.float64, 3))
        with pytest.raises(rrf.RRFError) as e:
            p.panel_qr(Y)
        assert e.value.status == -6
        Vt = to_dev(oracle.geqr2(W.random_dense(1024, 32, np.float64, 4))[0])
        Tt = to_dev(np.triu(W.random_dense(32, 32, np.float64, 5)))
        X = to_dev(W.random_dense(1024, 8, np.float64, 6))
        with pytest.raises(rrf.RRFError) as e:
            p.apply_block_reflector(Vt, Tt, X)
        assert e.value.status == -6
    monkeypatch.delenv("RRF_TEST_SPIN_LIMIT")
    _check_against_live_oracle(w, A)


def test_deterministic_repeat():
    w = W.scaled("galore_fp32_4096x4096", 1024, 768)
    A = to_dev(W.build_matrix(w))
    with rrf.Plan(torch.float32, 1024, 768, w.block_b) as p:
        Q1, B1, k1 = p.run(A, w.tol, w.block_b, w.sketch_seed)
        Q2, B2, k2 = p.run(A, w.tol, w.block_b, w.sketch_seed)
        torch.cuda.synchronize()
        assert k1 == k2
        assert torch.equal(Q1, Q2) and torch.equal(B1, B2)


def test_nonfinite_input_is_an_error():
    A = W.random_dense(64, 48, np.float64, 9)
    A[5, 7] = np.nan
    with rrf.Plan(torch.float64, 64, 48, 16) as p:
        with pytest.raises(rrf.RRFError) as e:
            p.run(to_dev(A), 1e-3, 16, 1)
        assert e.value.status == -3


def test_caller_provided_workspace():
    # rrf_plan_create_in: every device buffer carved from a workspace the
    # caller allocated (here a torch tensor); results bit-identical to a plan
    # that allocates its own, Q and B inside the workspace, and two runs in a
    # row reuse it.
    w = W.scaled("galore_fp32_4096x4096", 1024, 768)
    A = to_dev(W.build_matrix(w))
    need = rrf.workspace_size(torch.float32, 1024, 768, 32)
    ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    off = (-ws.data_ptr()) % 256
    ws = ws[off:off + need]
    with rrf.Plan(torch.float32, 1024, 768, 32) as p:
        Q1, B1, k1 = p.run(A, w.tol, 32, w.sketch_seed)
    with rrf.Plan(torch.float32, 1024, 768, 32, workspace=ws) as p:
        Qr, _, _, Br, _, _ = p.run_raw(A, w.tol, 32, w.sketch_seed)
        lo, hi = ws.data_ptr(), ws.data_ptr() + need
        assert lo <= Qr < hi and lo <= Br < hi
        Q2, B2, k2 = p.run(A, w.tol, 32, w.sketch_seed)
        torch.cuda.synchronize()
        assert k1 == k2
        assert torch.equal(Q1, Q2) and torch.equal(B1, B2)
    with pytest.raises(rrf.RRFError) as e:
        rrf.Plan(torch.float32, 1024, 768, 32, workspace=ws[:need - 256])
    assert e.value.status == -1


@pytest.mark.parametrize("nth", [1, 13, 25, 26])
def test_allocation_failure_is_reported(monkeypatch, nth):
    # RRF_FAULT_ALLOC=N fails the plan's N-th allocation (25 device buffers
    # for a binary64 plan, then the pinned run state): rrf_plan_create
    # returns RRF_ERR_NOMEM, frees what it had, and a later plan works.
    monkeypatch.setenv("RRF_FAULT_ALLOC", str(nth))
    say(f"allocation failure {nth}")
    with pytest.raises(rrf.RRFError) as e:
        rrf.Plan(torch.float64, 500, 300, 16)
    assert e.value.status == -4
    monkeypatch.delenv("RRF_FAULT_ALLOC")
    w = W.WORKLOADS["tiny_fp64_500x300"]
    with rrf.Plan(torch.float64, 500, 300, 16) as p:
        _, _, k = p.run(to_dev(W.build_matrix(w)), w.tol, 16, w.sketch_seed)
    assert k == _oracle(w, W.build_matrix(w)).k


def test_input_is_not_modified():
    w = W.scaled("square_fp64_16384", 512, 512)
    A = to_dev(W.build_matrix(w))
    A0 = A.clone()
    with rrf.Plan(torch.float64, 512, 512, 64) as p:
        p.run(A, w.tol, w.block_b, w.sketch_seed)
    torch.cuda.synchronize()
    assert torch.equal(A, A0)


def test_padded_leading_dimension():
    w = W.scaled("tiny_fp64_500x300", 300, 200)
    A = W.build_matrix(w)
    big = torch.zeros((310, 200), dtype=torch.float64, device="cuda")
    big = big.t().contiguous().t()
    big[:300] = torch.from_numpy(A).cuda()
    view = big[:300]          # lda = 310
    assert view.stride() == (1, 310)
    with rrf.Plan(torch.float64, 300, 200, 16) as p:
        Q, B, k = p.run(view, w.tol, w.block_b, w.sketch_seed)
    ref = oracle.hbarrf(A, w.tol, w.block_b, w.sketch_seed)
    assert k == ref.k


def _golden():
    if not os.path.exists(GOLDEN):
        return {}
    with open(GOLDEN) as f:
        return json.load(f)["configs"]


@pytest.mark.parametrize("name", W.CONFIGS)
def test_full_size_config_against_stored_oracle(name):
    g = _golden().get(name)
    if g is None:
        pytest.skip("oracle value not stored for this workload")
    w = W.WORKLOADS[name]
    say(f"full-size {name}: building A")
    A = W.build_matrix(w)
    Ad = to_dev(A)
    del A
    say(f"full-size {name}: rrf_run")
    with rrf.Plan(_tdt(w.dtype), w.m, w.n, w.block_b) as p:
        Q, B, k = p.run(Ad, w.tol, w.block_b, w.sketch_seed)
        tr = p.trace()
    assert k == g["k"]
    orth, res = gpu_metrics_torch(Ad, Q, B)
    dt = np.dtype(w.dtype)
    assert orth <= ORTH_TOL[dt]
    assert res <= residual_bound(g["residual_rel"], dt)
    # The guarantee of Alg. 2 holds at any size.
    assert res <= w.tol * (1 + 1e-6)
    # Theorem 3.1 at full size: Q^T A Omega[:, :k] is upper triangular.
    Om = torch.from_numpy(oracle.normal_v1(w.sketch_seed, w.n, 0, k, dtype=dt)).cuda()
    R = Q.t().contiguous().to(torch.float64) @ (Ad.to(torch.float64) @ Om.to(torch.float64))
    low = torch.tril(R, -1).abs().max().item()
    assert low <= 1e3 * np.finfo(dt).eps * R.abs().max().item()
    assert tr["nblocks"] == g["blocks"]


def test_log_and_stop_mode_environment(monkeypatch, capfd):
    # RRF_LOG=1: one stderr line per run and one per block; RRF_STOP_MODE
    # selects the initial stop mode (subtract here, same k as the oracle's).
    monkeypatch.setenv("RRF_LOG", "1")
    monkeypatch.setenv("RRF_STOP_MODE", "subtract")
    w = W.scaled("square_fp64_16384", 1024, 800, block_b=32, tol=1e-4)
    A = W.build_matrix(w)
    ref = oracle.hbarrf(A, w.tol, w.block_b, w.sketch_seed, stop="subtract")
    with rrf.Plan(torch.float64, 1024, 800, 32) as p:
        _, _, k = p.run(to_dev(A), w.tol, 32, w.sketch_seed)
        tr = p.trace()
    assert k == ref.k
    err = capfd.readouterr().err
    assert f"-> k={k} blocks={tr['nblocks']}" in err and "mode=1" in err
    assert err.count("rrf_run:   block") == tr["nblocks"]
