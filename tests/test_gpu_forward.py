"""GPU parity of the decomposed forward (HIP path through the C ABI) against
the float64 oracle, and decomposed against undecomposed.

Tolerances
  * fp32 inputs: max |O - O_f64| <= 1e-5 (required for the fp32 exactness case).
  * 16-bit inputs: max |O - O_f64| <= 1e-2 (required) everywhere, including
    near one-hot rows, and a relative-L2 bound derived from the arithmetic: P
    is rounded to the input type before the PV product (unit roundoff 2^-8
    for bf16, 2^-11 for fp16) and O is normalised by the sum of the rounded
    weights, which gives rel-L2 of order 1e-3 (bf16) / 2e-4 (fp16); the tests
    allow 4e-3 / 6e-4.
  * LSE uses fp32 statistics only: |LSE - LSE_f64| <= 1e-4 (16-bit scores are
    exact products accumulated in fp32).
  * decomposed vs undecomposed (depth 0) on the same inputs: rel-L2 <= 1e-3.
"""
import numpy as np
import pytest
import torch

from oracle import dense
from oracle import planner as oplan
from paper_2604_20819_amd import synth
from tests.gpu_util import need_gpu, rel_l2, run_forward, say

pytestmark = pytest.mark.gpu

REL = {"bf16": 4e-3, "f16": 6e-4, "f32": 1e-6}


def _check_vs_oracle(O, LSE, Q, K, V, causal, dt, rows=None, atol=None):
    Of, LSEf = dense.attention_forward(synth.as_f64(Q), synth.as_f64(K), synth.as_f64(V),
                                       causal, rows=rows)
    if rows is None:
        Og, LSEg = O.double().numpy(), LSE.double().numpy()
    else:
        Og = np.stack([O[:, r, h].double().numpy() for h, r in enumerate(rows)], axis=2)
        LSEg = np.stack([LSE[:, h, r].double().numpy() for h, r in enumerate(rows)], axis=1)
    err = np.abs(Og - Of).max()
    rl = rel_l2(Og, Of)
    lerr = np.abs(LSEg - LSEf).max()
    say(f"max_abs={err:.3e} rel_l2={rl:.3e} lse_abs={lerr:.3e}")
    assert np.isfinite(Og).all() and np.isfinite(LSEg).all()
    if atol is not None:
        assert err <= atol
    elif dt == "f32":
        assert err <= 1e-5
    else:
        assert err <= 1e-2
    assert rl <= REL[dt]
    assert lerr <= 1e-4
    return rl


def test_fp32_exactness_case():
    """B=1, H=1, d=64, L=1024, non-causal, fp32, depth 1 forced, all rows."""
    need_gpu()
    say("fp32 L=1024 H=1 d=64 depth=1")
    Q, K, V = synth.make_inputs(20819 + 1, 1, 1024, 1, 64, "f32")
    O, LSE, plan = run_forward(Q, K, V, causal=False, depth=1)
    assert plan.depth == 1 and plan.num_tasks == 7
    _check_vs_oracle(O, LSE, Q, K, V, False, "f32")


GRID = [(dt, d, causal, L, depth)
        for dt in ("bf16", "f16") for d in (64, 128) for causal in (False, True)
        for L, depth in ((1, 0), (1, 1), (100, 1), (1000, 0), (1000, 1), (2049, 2))]


@pytest.mark.parametrize("dt,d,causal,L,depth", GRID)
def test_small_grid_vs_oracle(dt, d, causal, L, depth):
    need_gpu()
    say(f"grid dt={dt} d={d} causal={causal} L={L} depth={depth}")
    Q, K, V = synth.make_inputs(7 + L + d, 2, L, 3, d, dt)
    O, LSE, plan = run_forward(Q, K, V, causal, depth=depth)
    assert plan.depth == depth
    _check_vs_oracle(O, LSE, Q, K, V, causal, dt)


HEAD_DIMS = [32, 96, 160, 192, 224, 256]


@pytest.mark.parametrize("d", HEAD_DIMS)
@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
def test_other_head_dims(d, dt):
    """Sec. 5 (kernel coverage): the forward covers head dims 32 to 256.  Rows
    of the K/V tiles are padded in LDS; the padding must never reach O.  A
    ragged length, causal and non-causal, undecomposed and decomposed.

    Early causal rows average a few keys; O is normalised by the sum of the
    rounded weights it was built from, so they too stay within the flat
    1e-2 max-abs bound."""
    need_gpu()
    for causal, L, depth in ((False, 700, 0), (True, 1150, 1), (False, 333, 2)):
        say(f"head dim d={d} dt={dt} causal={causal} L={L} depth={depth}")
        Q, K, V = synth.make_inputs(13 + d + L, 1, L, 3, d, dt)
        O, LSE, plan = run_forward(Q, K, V, causal, depth=depth)
        assert plan.depth == depth
        _check_vs_oracle(O, LSE, Q, K, V, causal, dt)


@pytest.mark.parametrize("d,causal", [(64, True), (128, False)])
def test_fp32_grid(d, causal):
    need_gpu()
    for L, depth in ((77, 0), (700, 1), (1500, 2)):
        say(f"fp32 grid d={d} causal={causal} L={L} depth={depth}")
        Q, K, V = synth.make_inputs(11 + L, 1, L, 2, d, "f32")
        O, LSE, _ = run_forward(Q, K, V, causal, depth=depth)
        _check_vs_oracle(O, LSE, Q, K, V, causal, "f32")


@pytest.mark.parametrize("dt,causal", [("bf16", False), ("bf16", True), ("f16", True)])
def test_decomposed_matches_undecomposed(dt, causal):
    need_gpu()
    say(f"decomposed vs undecomposed dt={dt} causal={causal}")
    Q, K, V = synth.make_inputs(99, 1, 4100, 4, 128, dt)
    O0, L0, _ = run_forward(Q, K, V, causal, depth=0)
    for depth in (1, 2, 3):
        O1, L1, _ = run_forward(Q, K, V, causal, depth=depth)
        r = rel_l2(O1.numpy(), O0.numpy())
        say(f"depth {depth}: rel_l2 vs depth 0 = {r:.3e}")
        assert r <= 1e-3
        assert np.abs(L1.numpy() - L0.numpy()).max() <= 1e-5


LEVEL_CASES = [([(13, (0, 1, 3, 9))], 1), ([(21, (0, 1, 4, 14, 16))], 1),
               ([(13, (0, 1, 3, 9))], 2), ([(7, (0, 1, 3)), (13, (0, 1, 3, 9))], 2),
               ([(13, (0, 1, 3, 9)), (7, (0, 1, 3))], 2),
               ([(3, (0, 1)), (7, (0, 1, 3)), (3, (0, 1))], 3)]


@pytest.mark.parametrize("levels,depth", LEVEL_CASES,
                         ids=["c13", "c21", "c13x2", "c7-c13", "c13-c7", "c3-c7-c3"])
@pytest.mark.parametrize("causal", [False, True])
def test_other_interest_sets_and_mixed_levels(levels, depth, causal):
    """Section 3.3: any valid interest set (App. C, Table "interest_set"), and
    a different one per depth.  The plan's tasks are the oracle planner's; the
    output matches the float64 oracle and the undecomposed call."""
    need_gpu()
    L = 3000
    Q, K, V = synth.make_inputs(77 + depth, 1, L, 3, 128, "bf16")
    say(f"interest sets {levels} depth {depth} causal={causal}")
    O0, L0, _ = run_forward(Q, K, V, causal, depth=0)
    O, LSE, plan = run_forward(Q, K, V, causal, depth=depth, levels=levels)
    full = (levels + [levels[-1]] * depth)[:depth]
    ref_tasks = oplan.build_tasks_levels(L, full)
    assert plan.num_tasks == len(ref_tasks)
    for t in (0, len(ref_tasks) // 2, len(ref_tasks) - 1):
        assert plan.task(t)["runs"] == oplan.runs(ref_tasks[t])
    _check_vs_oracle(O, LSE, Q, K, V, causal, "bf16")
    r = rel_l2(O.numpy(), O0.numpy())
    say(f"  rel_l2 vs depth 0 = {r:.3e}")
    assert r <= 1e-3
    assert np.abs(LSE.numpy() - L0.numpy()).max() <= 1e-5


@pytest.mark.parametrize("causal", [False, True])
def test_launch_groupings_agree(causal):
    """Slot counts and tasks per launch group change only the order of the
    exact power-of-two-scaled merge sums: results agree to fp32 rounding,
    and each matches the oracle."""
    need_gpu()
    Q, K, V = synth.make_inputs(5, 1, 3000, 2, 128, "bf16")
    ref = None
    for depth, n_slots, tps in ((2, 1, 0), (2, 3, 0), (2, 2, 1), (2, 2, 5), (2, 1, 32),
                                (1, 2, 7), (1, 1, 2), (1, 3, 3)):
        say(f"groups causal={causal} depth={depth} n_slots={n_slots} tasks_per_slot={tps}")
        O, LSE, plan = run_forward(Q, K, V, causal, depth=depth, n_slots=n_slots,
                                   tasks_per_slot=tps)
        if tps:
            assert plan.tasks_per_slot == tps
        if ref is None:
            ref = (O, LSE)
            _check_vs_oracle(O, LSE, Q, K, V, causal, "bf16")
            continue
        r = rel_l2(O.numpy(), ref[0].numpy())
        say(f"  rel_l2 vs first grouping = {r:.3e}")
        assert r <= 2e-5
        assert np.abs(LSE.numpy() - ref[1].numpy()).max() <= 1e-5


def test_overflowing_scores_stay_finite():
    """Scores of order 200 (lse far above ln(FLT_MAX) ~ 88.72): the max-shifted
    path must stay finite and exact (App. A.1)."""
    need_gpu()
    say("overflow scores")
    Q, K, V = synth.make_inputs(3, 1, 1500, 2, 128, "bf16")
    Q = (Q.float() * 4).to(torch.bfloat16)
    K = (K.float() * 4).to(torch.bfloat16)
    for depth in (0, 1, 2):
        O, LSE, _ = run_forward(Q, K, V, False, depth=depth)
        assert LSE.max().item() > 88.72
        # near one-hot softmax rows: the dominant weight is rounded to bf16
        # like every other, and O is normalised by the sum of the rounded
        # weights, so a one-hot row returns its V row and the flat bound holds
        _check_vs_oracle(O, LSE, Q, K, V, False, "bf16")


@pytest.mark.parametrize("dt,causal", [("bf16", False), ("f16", True)])
def test_rising_scores_take_the_exact_maximum_again(dt, causal):
    """Scores that climb by about 9 (log2 units) from one 64-key tile to the
    next: a tile that keeps the row's shift finds weights far above the 2^16
    bound on most tiles, recomputes its scores and takes the exact maximum;
    the result must still match float64 (App. A.1), at depths 0-2."""
    need_gpu()
    B, L, H, d = 1, 1536, 2, 64
    Q, K, V = synth.make_inputs(77, B, L, H, d, dt)
    e = torch.ones(d, dtype=torch.float32) / d ** 0.5
    ramp = (torch.arange(L, dtype=torch.float32) // 64) * 20.0   # per tile: +20 along e
    Q = (Q.float() + 3.0 * e).to(Q.dtype)
    K = (K.float() + ramp[None, :, None, None] * e).to(K.dtype)
    Qf, Kf = synth.as_f64(Q), synth.as_f64(K)
    s = np.einsum("blhd,bmhd->bhlm", Qf, Kf) / np.sqrt(d) * np.log2(np.e)
    step = np.median(s[..., 64:128].max(-1) - s[..., :64].max(-1))
    assert step > 8          # the bound's 16 doublings are gone within two tiles
    for depth in (0, 1, 2):
        say(f"rising scores dt={dt} causal={causal} depth={depth}")
        O, LSE, _ = run_forward(Q, K, V, causal, depth=depth)
        _check_vs_oracle(O, LSE, Q, K, V, causal, dt)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_one_hot_rows_return_the_value_row(dt):
    """Scores so peaked that every softmax row is one-hot to far below fp32
    resolution: O must be the V row of the row's own key (Q = K scaled, all
    keys distinct), up to a few fp32 roundings, at depths 0-2."""
    need_gpu()
    L, H, d = 777, 2, 64
    Q, K, V = synth.make_inputs(41, 1, L, H, d, dt)
    K = (Q.float() * 8).to(Q.dtype)   # s_ii = 8|q_i|^2 / sqrt(d) dominates s_ij
    Q = (Q.float() * 8).to(Q.dtype)
    Qf, Kf = synth.as_f64(Q), synth.as_f64(K)
    s = np.einsum("blhd,bmhd->bhlm", Qf, Kf) / np.sqrt(d)
    top2 = np.sort(s, axis=-1)[..., -2:]
    assert (np.argmax(s, axis=-1) == np.arange(L)).all()
    assert (top2[..., 1] - top2[..., 0]).min() > 30   # e^-30 ~ 1e-13
    want = synth.as_f64(V)
    for depth in (0, 1, 2):
        say(f"one-hot rows dt={dt} depth={depth}")
        O, LSE, _ = run_forward(Q, K, V, False, depth=depth)
        err = float(np.abs(O.double().numpy() - want).max())
        say(f"  max |O - V| = {err:.3e}")
        assert err <= 8 * 2.0 ** -24 * float(np.abs(want).max())


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_host_resident_streamed_small(dt):
    need_gpu()
    say(f"host streamed small {dt}")
    Q, K, V = synth.make_inputs(17, 2, 3001, 2, 64, dt)
    O, LSE, plan = run_forward(Q, K, V, True, depth=2, host=True)
    assert plan.depth == 2
    _check_vs_oracle(O, LSE, Q, K, V, True, dt)
    Od, Ld, _ = run_forward(Q, K, V, True, depth=2)
    assert rel_l2(O.numpy(), Od.numpy()) <= 1e-6


def test_bf16_L32768_single_level():
    """B=1, H=16, d=128, L=32768, non-causal bf16, depth 1: 2048 sampled rows
    per head against float64; all rows against the undecomposed kernel."""
    need_gpu()
    say("bf16 L=32768 H=16 depth 1")
    B, L, H, d = 1, 32768, 16, 128
    Q, K, V = synth.make_inputs(20819 + 2, B, L, H, d, "bf16")
    O, LSE, plan = run_forward(Q, K, V, False, depth=1)
    assert plan.depth == 1 and plan.num_tasks == 7
    rows = synth.sample_rows(20819 + 2, L, 2048, H)
    _check_vs_oracle(O, LSE, Q, K, V, False, "bf16", rows=rows)
    O0, L0, _ = run_forward(Q, K, V, False, depth=0)
    r = rel_l2(O.numpy(), O0.numpy())
    say(f"rel_l2 vs depth 0 = {r:.3e}")
    assert r <= 1e-3
