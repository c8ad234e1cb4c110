"""Algorithm 1 per arrival on the GPU against the oracle, through the C ABI
(needs an MI355X).

Each request is scored against the state the requests before it left.  The
oracle runs the same schedule following the GPU's placement wherever its own
decision is near a boundary (rounding may decide it) and the two differ, after
checking that placement is capacity-eligible; so both sides go on from the
same state and every request is compared.  Same bar as the window kernel:
hits, choices and flags exact except on near-boundary decisions (counted and
capped), |A| and |C| exact, |T| within the candidates rounding may move,
TTFT/TPOT within 1e-5 relative; then the final state, the refused-block count
and a snapshot scored afterwards.
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import (DeviceWindow, compare_decisions, compare_sequential, edge_window,
                            load_window, reqs_of)
from tests.tinywin import chain_hashes, make_window

pytestmark = pytest.mark.gpu

SIMPLE_ALPHA = [0.02, 1e-3, 1e-6, 1e-6, 1e-5, 2e-9]


@pytest.fixture(scope="module")
def ps():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_33224_amd as ps
    return ps


@pytest.fixture()
def scorer(ps):
    s = ps.Scorer(0)
    yield s
    s.close()


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _states_equal(o, scorer, label):
    so, sg = o.state(), scorer.state()
    for k in ("D", "Q", "P", "S", "set_size"):
        bad = np.nonzero(so[k] != sg[k])[0]
        assert len(bad) == 0, f"{label}: {k} differs at instances {bad[:5]}"


def _schedule_check(ps, scorer, w, label, budget=None, follow=True, **policy):
    """Schedule w on both sides and compare every request, the final state
    and (follow) a snapshot scored afterwards.  Returns (near-boundary
    count, results)."""
    load_window(scorer, w, **policy)
    if budget:
        scorer.set_schedule_budget(budget)
    dw = DeviceWindow(w)
    res, sizes, dropped = dw.schedule(scorer)
    o = oracle.Oracle.from_window(w)
    od, dropped_o = o.window_schedule(w, follow=res["instance"], **policy)
    nb = compare_sequential(res, sizes, od, label=label)
    assert dropped == dropped_o, f"{label}: dropped {dropped} vs {dropped_o}"
    _states_equal(o, scorer, label)
    if follow and w.n_req:
        # the derived data the window kernel reads was rebuilt: score the
        # same requests against the final state
        res2, sizes2 = dw.score(scorer)
        od2 = o.window_score(w, **policy)
        compare_decisions(res2, sizes2, od2, label=f"{label} then snapshot")
    return nb, res


@pytest.mark.parametrize("name,policy", [("c1", {}), ("c1", dict(tpot_slo=0.030, b_max=96)),
                                         ("c2", {}), ("c2_50", {})])
def test_schedule_full_window(ps, scorer, name, policy):
    _say(f"schedule parity {name} {policy}")
    w = synth.generate(name)
    nb, res = _schedule_check(ps, scorer, w, f"{name} {policy}", **policy)
    _say(f"{name}: {w.n_req} compared, {nb} near-boundary")
    # the sizes path and the results are deterministic
    load_window(scorer, w, **policy)
    res2, _, _ = DeviceWindow(w).schedule(scorer, with_sizes=False)
    assert res2.tobytes() == res.tobytes()


@pytest.mark.parametrize("name,n", [("c3", 4096), ("c4", 8192), ("c5", 8192)])
def test_schedule_leading_slice(ps, scorer, name, n):
    """The first n arrivals of the full-size windows, per arrival on both
    sides against the full-size snapshot, then the state after the slice."""
    _say(f"schedule parity {name} first {n}: generating")
    w = synth.generate(name).subset(range(n))
    nb, res = _schedule_check(ps, scorer, w, f"{name} first {n}")
    _say(f"{name} first {n}: compared, {nb} near-boundary, "
         f"{int((res['flags'] & ps.PS_R_FALLBACK != 0).sum())} fallback")


def test_schedule_round_robin_closed_form(ps, scorer):
    """Identical instances (D = 3), fresh chains, B_max = 7: request k goes
    to instance k mod 5 and the last 3 of 23 are rejected."""
    chains = [chain_hashes(4, base=10_000 * (k + 1)) for k in range(23)]
    w = make_window([[] for _ in range(5)], chains, [3] * 5, [0] * 5, [0] * 5, [0] * 5,
                    np.float32(SIMPLE_ALPHA), (64,), np.float32([[0.01, 0.0, 0.0]]),
                    np.float32([1.0]), cap=64, tpot_slo=10.0, b_max=7, kv_cap_tokens=10**9)
    _, res = _schedule_check(ps, scorer, w, "round robin")
    assert list(res["instance"]) == [k % 5 for k in range(20)] + [-1] * 3
    assert (res["flags"][20:] == ps.PS_R_REJECT).all()


@pytest.mark.parametrize("budget_rows", [1, 7, 64])
def test_schedule_split_into_launches(ps, scorer, budget_rows):
    """A hit budget smaller than the window splits it into launches; the
    results are those of one launch."""
    w = synth.generate("c1", n_req=600)
    load_window(scorer, w)
    ref, ref_sizes, ref_drop = DeviceWindow(w).schedule(scorer)
    _, res = _schedule_check(ps, scorer, w, f"budget {budget_rows} rows",
                             budget=budget_rows * w.n_inst * 4)
    assert res.tobytes() == ref.tobytes()


def test_schedule_edge_instance_counts(ps, scorer):
    """Pool sizes around the wave and workgroup widths (one thread owning
    several instances above 512), part of the pool at its batch limit."""
    for n_inst in (1, 63, 64, 65, 100, 257, 513, 1000, 2100):
        ch = chain_hashes(300, base=17)
        rng = np.random.default_rng(n_inst)
        sets = [ch[:int(rng.integers(0, 300))] for _ in range(n_inst)]
        chains = [ch[:k] for k in (1, 2, 65, 150, 300, 299, 40)]
        chains += [(ch[:100], chain_hashes(5, base=10**9 + j)) for j in range(6)]
        chains += [ch[:k] + chain_hashes(3, base=2 * 10**9 + k) for k in (10, 200, 290)]
        for b_max in (512, 40):
            _say(f"edge n_inst={n_inst} b_max={b_max}")
            w = edge_window(sets, chains, b_max=b_max, cap=400)
            _schedule_check(ps, scorer, w, f"n_inst={n_inst} b_max={b_max}")


def test_schedule_sessions_follow_their_blocks(ps, scorer):
    """Requests that extend an earlier request's chain find its blocks on
    the instance it went to (hit extensions within one launch), including
    chains longer than the LDS stage and split descriptors."""
    rng = np.random.default_rng(3)
    sess = [chain_hashes(int(n), base=10**7 * (k + 1)) for k, n in
            enumerate(rng.integers(50, 1500, 12))]
    chains = []
    for step in range(6):
        for s in sess:
            k = min(len(s), 40 + step * 250)
            chains.append((s[:k // 2], s[k // 2:k]) if step % 2 else s[:k])
    sets = [sess[k % 12][:int(rng.integers(0, 30))] for k in range(20)]
    w = edge_window(sets, chains, cap=4000, eta=0.2)
    _, res = _schedule_check(ps, scorer, w, "sessions")
    assert (res["hit_blocks"][12:] > 0).mean() > 0.5


def test_schedule_cap_refuses_blocks(ps, scorer):
    w = synth.generate("c1", n_req=1024, cap=1100)
    _schedule_check(ps, scorer, w, "cap 1100")


def test_schedule_duplicates_zero_cost_and_empty(ps, scorer):
    ch = chain_hashes(200, base=3)
    other = chain_hashes(50, base=7 * 10**6)
    sets = [ch[:50] + ch[:50] + other, ch[1:150], ch[:10] + ch[11:200], ch[:100][::-1]]
    chains = [ch, ch[:120], other, [], ch[:1], ch + ch[:5], other + other]
    _schedule_check(ps, scorer, edge_window(sets, chains, cap=600), "dups/holes")
    w = edge_window(sets, chains, cap=600)
    w.alpha = np.float32([0.02, 0.0, 1e-6, 0.0, 0.0, 0.0])  # Z = 0: all of A is kept
    for eta in (0.0, 0.3):
        _schedule_check(ps, scorer, w, f"Z=0 eta={eta}", eta=eta)


SELECTORS = ["DCQ", "D", "DQ", "DC", "DQC", "HCQ", "RANDOM", "LMETRIC"]
LAYERS = {"G": 2 | 4, "C": 4, "T": 2 | 8, "CT": 8, "F": 0}


@pytest.mark.parametrize("name,gen", [("c1", dict(n_req=512)),
                                      ("c3", dict(n_inst=128, n_sess=256, n_req=512))])
def test_schedule_selectors_and_layers(ps, scorer, name, gen):
    w = synth.generate(name, **gen)
    for k, sel in enumerate(SELECTORS):
        for layer, fl in LAYERS.items():
            pol = dict(flags=fl | (k << 8), rand_seed=7654321 + k)
            _schedule_check(ps, scorer, w, f"{name} {sel} {layer}", follow=False, **pol)


@pytest.mark.parametrize("name,policy", [("c1", dict(tpot_slo=0.030, b_max=96)), ("c2", {})])
def test_replay_snapshot_placements(ps, scorer, name, policy):
    """The oracle's snapshot placements replayed in arrival order on both
    sides: hits exact, latencies within 1e-5, same final state."""
    _say(f"replay {name}")
    w = synth.generate(name)
    o = oracle.Oracle.from_window(w)
    snap = o.window_score(w, **policy)
    hit, ttft, tpot, dropped_o = o.window_replay(w, snap.inst, **policy)
    load_window(scorer, w, **policy)
    res, dropped = DeviceWindow(w).replay(scorer, snap.inst)
    placed = snap.inst >= 0
    assert (res["instance"] == snap.inst).all()
    assert (res["hit_blocks"][placed] == hit[placed]).all()
    assert (res["flags"][~placed] == ps.PS_R_REJECT).all()
    for nm, ref in (("ttft", ttft), ("tpot", tpot)):
        g = res[nm][placed].astype(np.float64)
        rel = np.abs(g - ref[placed]) / np.maximum(np.abs(ref[placed]), 1e-30)
        assert rel.max() <= 1e-5, f"{name}: replay {nm} rel err {rel.max():.3g}"
    assert dropped == dropped_o
    _states_equal(o, scorer, f"replay {name}")


def test_schedule_invalid_descriptor_and_errors(ps, scorer):
    import torch
    w = synth.generate("c1", n_req=16)
    load_window(scorer, w)
    reqs = reqs_of(w)
    reqs["pre_off"][3] = len(w.pool) + 5
    reqs["tail_len"][5] = -1
    d_pool = ps.to_device_u64(w.pool)
    d_reqs = ps.to_device_bytes(reqs)
    d_out = torch.zeros(16 * 20, dtype=torch.uint8, device="cuda")
    scorer.schedule_dev(d_pool, len(w.pool), d_reqs, 16, d_out)
    res = ps.results_from_device(d_out)
    assert res["flags"][3] == ps.PS_R_INVALID and res["flags"][5] == ps.PS_R_INVALID
    assert res["instance"][3] == -1
    # the other 14 are those of a window without the two malformed entries
    keep = [k for k in range(16) if k not in (3, 5)]
    o = oracle.Oracle.from_window(w)
    od, _ = o.window_schedule(w.subset(np.array(keep)), follow=res["instance"][keep])
    compare_sequential(res[keep], None, od, label="invalid")
    _states_equal(o, scorer, "invalid")
    # an empty window changes nothing
    before = scorer.state()
    assert scorer.schedule_dev(d_pool, len(w.pool), d_reqs, 0, d_out) == 0
    after = scorer.state()
    assert all((before[k] == after[k]).all() for k in before)
    # a replay entry outside [-1, n_inst) is refused before any change
    d_inst = torch.full((16,), w.n_inst, dtype=torch.int32, device="cuda")
    with pytest.raises(ps.PackServeError) as e:
        scorer.replay_dev(d_pool, len(w.pool), d_reqs, 16, d_inst, d_out)
    assert e.value.code == ps.binding.PS_E_RANGE
    after2 = scorer.state()
    assert all((after[k] == after2[k]).all() for k in after)
    # B_max that would let a queue counter pass its 12-bit limit
    load_window(scorer, w, b_max=8000)
    with pytest.raises(ps.PackServeError) as e:
        scorer.schedule_dev(d_pool, len(w.pool), d_reqs, 16, d_out)
    assert e.value.code == ps.binding.PS_E_RANGE


# ------------------------------------------------------------ speculative batches
def _schedule_spec_and_full(ps, scorer, w, batch, **policy):
    """The window scheduled from the same loaded state with every request
    scored in full, then with speculative batches of `batch`: both runs'
    (results, sizes, dropped, final state, stats)."""
    runs = []
    for b in (0, batch):
        load_window(scorer, w, **policy)
        scorer.set_schedule_speculation(b)
        res, sizes, dropped = DeviceWindow(w).schedule(scorer)
        runs.append((res, sizes, dropped, scorer.state(), scorer.schedule_stats()))
    scorer.set_schedule_speculation(256)
    return runs


def _assert_same_schedule(runs, n_valid, label):
    (r0, s0, d0, st0, (f0, g0)), (r1, s1, d1, st1, (f1, g1)) = runs
    bad = np.nonzero(r0 != r1)[0]
    assert len(bad) == 0, f"{label}: {len(bad)} results differ, first request {bad[0]}"
    assert (s0 == s1).all(), f"{label}: set sizes differ at {np.nonzero((s0 != s1).any(1))[0][:5]}"
    assert d0 == d1, f"{label}: dropped {d0} vs {d1}"
    for k in st0:
        assert (st0[k] == st1[k]).all(), f"{label}: final {k} differs"
    assert (f0, g0) == (0, 0), f"{label}: without speculation the counts are {f0}, {g0}"
    assert f1 + g1 == n_valid, f"{label}: {f1} + {g1} decisions of {n_valid}"
    _say(f"{label}: identical; {f1} of {n_valid} decided from speculation")
    return f1


SPEC_WINDOWS = [("c1", {}, {}), ("c1", {}, dict(tpot_slo=0.030, b_max=96)),
                ("c2", dict(n_req=4096), {}), ("c2_50", dict(n_req=4096), {}),
                ("c3", dict(n_req=65536), {}), ("c4", dict(n_req=32768), {}),
                ("c5", dict(n_req=262144), {})]


@pytest.mark.parametrize("name,gen,policy", SPEC_WINDOWS)
def test_speculation_matches_full_scoring(ps, scorer, name, gen, policy):
    """Speculative batches decide exactly as scoring every request in full:
    results, set sizes, refused blocks and the final state byte for byte;
    most requests are decided from their speculative result."""
    w = synth.generate(name, **gen)
    if w.n_req > 4096:
        w = w.subset(range(2048))
    runs = _schedule_spec_and_full(ps, scorer, w, 256, **policy)
    n_spec = _assert_same_schedule(runs, w.n_req, f"{name} {policy}")
    assert n_spec > w.n_req // 2


@pytest.mark.parametrize("batch", [1, 2, 7, 64, 255])
def test_speculation_batch_sizes(ps, scorer, batch):
    w = synth.generate("c2", n_req=1500)
    _assert_same_schedule(_schedule_spec_and_full(ps, scorer, w, batch), w.n_req, f"batch {batch}")


def test_speculation_selectors_and_layers(ps, scorer):
    """Every keyed selector (Random and H-C-Q are always scored in full)
    with every admission layer, TTFT admission and the D-C-Q fallback."""
    w = synth.generate("c3", n_inst=128, n_sess=256, n_req=512)
    for k, sel in enumerate(SELECTORS):
        for layer, fl in list(LAYERS.items()) + [("F+TTFT", 1), ("F+DCQfb", 8 | 1)]:
            pol = dict(flags=fl | (k << 8), rand_seed=7654321 + k)
            runs = _schedule_spec_and_full(ps, scorer, w, 256, **pol)
            keyed = sel not in ("RANDOM", "HCQ")
            _assert_same_schedule(runs, w.n_req if keyed else 0, f"{sel} {layer}")


def test_speculation_edge_windows(ps, scorer):
    """Hit extensions inside a batch (sessions that follow their blocks),
    repeats and holes, Z = 0, the table cap, small and odd pool sizes."""
    rng = np.random.default_rng(3)
    sess = [chain_hashes(int(n), base=10**7 * (k + 1)) for k, n in
            enumerate(rng.integers(50, 1500, 12))]
    chains = []
    for step in range(6):
        for s in sess:
            k = min(len(s), 40 + step * 250)
            chains.append((s[:k // 2], s[k // 2:k]) if step % 2 else s[:k])
    sets = [sess[k % 12][:int(rng.integers(0, 30))] for k in range(20)]
    for batch in (256, 5):
        w = edge_window(sets, chains, cap=4000, eta=0.2)
        _assert_same_schedule(_schedule_spec_and_full(ps, scorer, w, batch, eta=0.2), w.n_req,
                              f"sessions batch {batch}")
    ch = chain_hashes(200, base=3)
    other = chain_hashes(50, base=7 * 10**6)
    sets = [ch[:50] + ch[:50] + other, ch[1:150], ch[:10] + ch[11:200], ch[:100][::-1]]
    chains = [ch, ch[:120], other, [], ch[:1], ch + ch[:5], other + other] * 3
    w = edge_window(sets, chains, cap=600)
    _assert_same_schedule(_schedule_spec_and_full(ps, scorer, w, 256), w.n_req, "dups/holes")
    w.alpha = np.float32([0.02, 0.0, 1e-6, 0.0, 0.0, 0.0])  # Z = 0: all of A is kept
    for eta in (0.0, 0.3):
        _assert_same_schedule(_schedule_spec_and_full(ps, scorer, w, 256, eta=eta), w.n_req,
                              f"Z=0 eta={eta}")
    w = synth.generate("c1", n_req=1024, cap=1100)
    _assert_same_schedule(_schedule_spec_and_full(ps, scorer, w, 256), w.n_req, "cap 1100")
    for n_inst in (1, 63, 65, 257, 2100):
        ch = chain_hashes(300, base=17)
        rng = np.random.default_rng(n_inst)
        sets = [ch[:int(rng.integers(0, 300))] for _ in range(n_inst)]
        chains = [ch[:k] for k in (1, 2, 65, 150, 300, 299, 40)] * 20
        for b_max in (512, 40):
            w = edge_window(sets, chains, b_max=b_max, cap=400)
            _assert_same_schedule(_schedule_spec_and_full(ps, scorer, w, 256, b_max=b_max),
                                  w.n_req, f"n_inst={n_inst} b_max={b_max}")


def test_speculation_setting_errors(ps, scorer):
    for bad in (-1, 257, 10**6):
        with pytest.raises(ps.PackServeError) as e:
            scorer.set_schedule_speculation(bad)
        assert e.value.code == ps.binding.PS_E_INVAL
    scorer.set_schedule_speculation(0)
    scorer.set_schedule_speculation(256)


def test_schedule_random_windows(ps, scorer):
    """100 of the seeded random windows scheduled per arrival: every
    request, the refused blocks and the final state against the oracle's
    schedule, a snapshot scored afterwards, and speculative batches of 64
    byte for byte against scoring every request in full."""
    from tests.test_gpu_parity import RANDOM_POLICIES, _random_window
    for seed in range(100):
        w = _random_window(seed)
        pol = RANDOM_POLICIES[seed % len(RANDOM_POLICIES)]
        label = f"random window {seed} ({w.n_inst} x {w.n_req}, {pol})"
        _say(label)
        _schedule_check(ps, scorer, w, label, **pol)
        _assert_same_schedule(_schedule_spec_and_full(ps, scorer, w, 64, **pol), w.n_req, label)
