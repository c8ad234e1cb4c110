"""GPU <-> oracle parity through the C ABI (needs an MI355X).

Bar: prefix hits and chosen instances bit-exact; flags and |A|, |C|, |T|
exact; predicted TTFT/TPOT within 1e-5 relative (fp32 vs fp64); decisions
whose oracle comparison lies within 1e-5 relative of a boundary are counted
and excluded from the exact check.
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import DeviceWindow, compare_decisions, gpu_model, load_window, reqs_of
from tests.gpu_util import edge_window as _edge
from tests.tinywin import chain_hashes, make_window

pytestmark = pytest.mark.gpu


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


# ------------------------------------------------------------- small windows
@pytest.mark.parametrize("name", ["c1", "c2"])
def test_hits_bit_exact_full_window(ps, scorer, name):
    _say(f"hits parity {name}")
    w = synth.generate(name)
    load_window(scorer, w)
    dw = DeviceWindow(w)
    got = dw.hits(scorer, w.n_inst)
    want = oracle.Oracle.from_window(w).window_hits(w)
    bad = np.argwhere(got != want)
    assert len(bad) == 0, f"{len(bad)} hits differ, first {bad[0]}: {got[tuple(bad[0])]} vs {want[tuple(bad[0])]}"


@pytest.mark.parametrize("name", ["c1", "c2", "c2_50"])
def test_decisions_full_window(ps, scorer, name):
    _say(f"decision parity {name}")
    w = synth.generate(name)
    load_window(scorer, w)
    dw = DeviceWindow(w)
    res, sizes = dw.score(scorer)
    od = oracle.Oracle.from_window(w).window_score(w)
    nb = compare_decisions(res, sizes, od, label=name)
    _say(f"{name}: {w.n_req} decisions, {nb} near-boundary excluded")
    # the path without set sizes (the benchmark's) decides identically
    res2, _ = dw.score(scorer, with_sizes=False)
    assert res2.tobytes() == res.tobytes()


def test_host_entry_point_matches_device(ps, scorer):
    w = synth.generate("c1")
    load_window(scorer, w)
    a = scorer.score(w.pool, reqs_of(w))
    b, _ = DeviceWindow(w).score(scorer)
    assert a.tobytes() == b.tobytes()


def test_deterministic(ps, scorer):
    w = synth.generate("c2", n_req=4096)
    load_window(scorer, w)
    dw = DeviceWindow(w)
    a, sa = dw.score(scorer)
    b, sb = dw.score(scorer)
    assert a.tobytes() == b.tobytes() and (sa == sb).all()


@pytest.mark.parametrize("policy", [dict(eta=0.0), dict(eta=1.0), dict(eta=0.25),
                                    dict(tpot_slo=1e-6), dict(tpot_slo=10.0),
                                    dict(flags=1), dict(flags=2), dict(flags=4), dict(flags=7),
                                    dict(b_max=1), dict(kv_cap_tokens=0)])
def test_policy_variants(ps, scorer, policy):
    _say(f"policy {policy}")
    w = synth.generate("c1")
    load_window(scorer, w, **policy)
    dw = DeviceWindow(w)
    res, sizes = dw.score(scorer)
    od = oracle.Oracle.from_window(w).window_score(w, **policy)
    compare_decisions(res, sizes, od, label=str(policy))
    res2, _ = dw.score(scorer, with_sizes=False)
    assert res2.tobytes() == res.tobytes()
    if policy.get("b_max") == 1 or policy.get("kv_cap_tokens") == 0:
        assert (res["instance"] == -1).all() and (res["flags"] == ps.PS_R_REJECT).all()
    if policy.get("tpot_slo") == 1e-6:
        assert ((res["flags"] & ps.PS_R_FALLBACK) != 0).all()


def test_non_monotone_model(ps, scorer):
    """Coefficients under which the zero-hit TPOT test is not one threshold
    on the request length (a negative context or quadratic term): the
    kernel scans the class in key order instead of using the thresholds."""
    for name, gen in (("c1", {}), ("c2", dict(n_req=2048))):
        w = synth.generate(name, **gen)
        w.beta = np.asarray(w.beta, np.float32).copy()
        w.beta[:, 2] = -2e-10
        w.alpha = np.asarray(w.alpha, np.float32).copy()
        w.alpha[3] = -1e-12
        load_window(scorer, w)
        dw = DeviceWindow(w)
        res, sizes = dw.score(scorer)
        od = oracle.Oracle.from_window(w).window_score(w)
        compare_decisions(res, sizes, od, label=f"{name} non-monotone")
        res2, _ = dw.score(scorer, with_sizes=False)
        assert res2.tobytes() == res.tobytes()


# ------------------------------------------------------------- edge windows
def _tail_only(w):
    """The same chains as tail segments only (no shared segment, so no
    prefix group): every request takes the scorer's per-request path.
    Needs each request's tail to follow its prefix in the pool."""
    assert (w.tail_off == w.pre_off + w.pre_len).all() or (w.tail_len == 0).all()
    t = w.subset(range(w.n_req))
    t.tail_off = w.pre_off.copy()
    t.tail_len = (w.pre_len + w.tail_len).astype(np.int32)
    t.pre_len = np.zeros_like(w.pre_len)
    return t


def _check_edge(ps, scorer, w, label, **policy):
    w.alpha = np.asarray(w.alpha, np.float32)
    load_window(scorer, w, **policy)
    o = oracle.Oracle.from_window(w)
    variants = [(w, label)]
    if (w.tail_off == w.pre_off + w.pre_len).all() and (w.pre_len > 0).any():
        variants.append((_tail_only(w), label + " tail-only"))
    first = None
    for v, lab in variants:
        dw = DeviceWindow(v)
        got = dw.hits(scorer, v.n_inst)
        want = o.window_hits(v)
        assert (got == want).all(), f"{lab}: hits differ at {np.argwhere(got != want)[:3]}"
        res, sizes = dw.score(scorer)
        od = o.window_score(v, **policy)
        compare_decisions(res, sizes, od, label=lab)
        res2, _ = dw.score(scorer, with_sizes=False)
        assert res2.tobytes() == res.tobytes(), f"{lab}: path without sizes differs"
        if first is None:
            first = res
        else:
            assert res.tobytes() == first.tobytes(), f"{lab}: differs from the grouped path"
    return first


def test_edge_single_instance_and_ragged_counts(ps, scorer):
    for n_inst in (1, 63, 100, 257, 1000):
        ch = chain_hashes(300, base=17)
        rng = np.random.default_rng(n_inst)
        sets = [ch[:int(rng.integers(0, 300))] for _ in range(n_inst)]
        chains = [ch[:k] for k in (1, 2, 65, 150, 300)] + [(ch[:100], chain_hashes(5, base=10**9))]
        _check_edge(ps, scorer, _edge(sets, chains), f"n_inst={n_inst}")
        # part of the pool at its batch limit: holders that are not eligible
        _check_edge(ps, scorer, _edge(sets, chains, b_max=40), f"n_inst={n_inst} b_max=40")


def test_edge_chain_lengths_around_stage(ps, scorer):
    ch = chain_hashes(5000, base=99)
    sets = [ch[:h] for h in (0, 1, 63, 64, 65, 1023, 1024, 1025, 2047, 4999, 5000)]
    chains = [ch[:k] for k in (1, 64, 1023, 1024, 1025, 2048, 5000)]
    # also split descriptors whose boundary falls inside the staged head
    chains += [(ch[:700], ch[700:3000]), (ch[:1], ch[1:1500])]
    _check_edge(ps, scorer, _edge(sets, chains), "stage")


def test_edge_hits_beyond_u16_slots(ps, scorer):
    """Hits above 65,533 blocks do not fit the scorer's 16-bit hit slots: the
    slot keeps an overflow mark and the hit is walked again where it is
    needed.  Chains of up to 70,000 blocks on instances holding 70,000,
    66,000, 65,534, 65,535 and 10 of them (grouped and tail-only)."""
    ch = chain_hashes(70000, base=31)
    sets = [ch[:70000], ch[:66000], ch[:65534], ch[:65535], ch[:10]]
    chains = [ch[:70000], ch[:65535], ch[:66001], ch[:65534], (ch[:30000], ch[30000:70000]),
              (ch[:8], ch[8:66500])]
    for eta in (0.5, 0.0):
        res = _check_edge(ps, scorer, _edge(sets, chains, cap=70000, D=[5, 9, 1, 2, 0],
                                            kv_cap_tokens=10**8), f"u16 overflow eta={eta}",
                          eta=eta)
    assert res["hit_blocks"].max() > 65533


def test_edge_fully_cached_and_empty_chain(ps, scorer):
    ch = chain_hashes(40, base=5)
    sets = [ch, ch[:20], []]
    res = _check_edge(ps, scorer, _edge(sets, [ch, [], ch[:1]]), "full/empty")
    assert res["hit_blocks"][0] in (40, 20, 0)


def test_edge_duplicates_and_non_prefix_closed(ps, scorer):
    ch = chain_hashes(200, base=3)
    other = chain_hashes(50, base=7 * 10**6)
    sets = [ch[:50] + ch[:50] + other,          # duplicates in the CSR row
            ch[1:150],                          # misses the first block
            ch[:10] + ch[11:200],               # hole at block 10
            ch[:100][::-1]]                     # order irrelevant
    _check_edge(ps, scorer, _edge(sets, [ch, ch[:120], other]), "dups/holes", )


def test_edge_zero_cache_benefit_and_eta(ps, scorer):
    ch = chain_hashes(64, base=11)
    sets = [ch[:h] for h in (0, 10, 20, 40, 64)]
    w = _edge(sets, [ch, ch[:32]])
    w.alpha = [0.02, 0.0, 1e-6, 0.0, 0.0, 0.0]   # Z = 0: all of A is kept
    _check_edge(ps, scorer, w, "Z=0", eta=0.0)
    for eta in (0.0, 0.3, 1.0):
        _check_edge(ps, scorer, _edge(sets, [ch, ch[:32]]), f"eta={eta}", eta=eta)


def test_edge_large_instance_count_uses_scratch(ps, scorer):
    n_inst = 20000
    ch = chain_hashes(128, base=23)
    rng = np.random.default_rng(1)
    sets = [ch[:int(h)] for h in rng.integers(0, 129, n_inst)]
    w = _edge(sets, [ch, ch[:64], ch[:1]], cap=128)
    res = _check_edge(ps, scorer, w, "n_inst=20000")
    assert not scorer.table_info()["hits_in_lds"]


# ------------------------------------------------------------- prefix groups
def _shared_pool_window(base=101, order_seed=0, **kw):
    """Requests sharing pool segments with different prefix lengths and
    their own tails (some cached after the segment), so that whichever
    request leads a group, members lie on both sides of its segment length.
    Segment S1's first block has more holders than a group record keeps,
    S2's has none, S3 has a zero hash inside."""
    rng = np.random.default_rng(base)
    S0 = chain_hashes(400, base=base)
    S1 = chain_hashes(120, base=base + 5 * 10**6)
    S2 = chain_hashes(40, base=base + 9 * 10**6)
    S3 = chain_hashes(30, base=base + 13 * 10**6)
    S3[5] = 0
    tails = [chain_hashes(int(rng.integers(1, 6)), base=base + 10**8 + 10**4 * k) for k in range(12)]
    pool = []

    def put(seq):
        off = len(pool)
        pool.extend(seq)
        return off

    o0, o1, o2, o3 = put(S0), put(S1), put(S2), put(S3)
    t_off = [put(t) for t in tails]
    n_inst = 26
    sets = [[] for _ in range(n_inst)]
    sets[0] = S0 + tails[0] + tails[1]      # all of S0, then tails 0 and 1
    sets[1] = S0[:120] + tails[2][:2]        # a shorter prefix, then tail 2's head
    sets[2] = S0[:50] + S0[60:100]           # a hole at block 50
    sets[3] = S0[:10] + tails[3]             # tail 3, reachable only after S0[:10]
    sets[4] = S0[:300]
    sets[5] = S0[1:200]                      # lacks the first block
    for i in range(6, 24):                   # 18 holders of S1's first block
        sets[i] = S1[:int(rng.integers(1, 121))]
    sets[6] += S0[:8]
    sets[7] += S3[:5] + S3[6:]
    sets[24] = S3[:5]
    sets[25] = S0[:399]
    reqs = []
    for k, p in enumerate([8, 9, 10, 11, 49, 50, 51, 100, 119, 120, 121, 200, 299, 300, 301,
                           398, 399, 400]):
        t = k % 4
        reqs.append((o0, p, t_off[t], len(tails[t])))
    reqs += [(o0, 10, t_off[3], len(tails[3])), (o0, 120, t_off[2], len(tails[2])),
             (o0, 400, t_off[0], len(tails[0])), (o0, 400, t_off[1], 0),
             (o0, 400, t_off[1], len(tails[1])), (o0, 300, t_off[0], 0)]
    reqs += [(o1, p, t_off[5], len(tails[5])) for p in (8, 60, 120)]
    reqs += [(o2, p, t_off[6], 1) for p in (8, 40)]
    reqs += [(o3, p, t_off[7], len(tails[7])) for p in (8, 30)]
    # no group: a short shared segment, a tail-only chain, an offset segment
    reqs += [(o0, 3, t_off[8], 2), (o0, 0, o0, 50), (o0 + 10, 30, t_off[9], 1), (o0 + 10, 30, t_off[9], 0)]
    perm = np.random.default_rng(order_seed).permutation(len(reqs))
    reqs = [reqs[k] for k in perm]
    return _edge(sets, None, pool=pool, reqs=reqs, cap=420, **kw)


def test_prefix_groups_shared_segments(ps, scorer):
    """Members of one group with segment lengths on both sides of the
    leader's, cached tails, holes, records without a result, zero hashes;
    several request orders (different leaders), policies and repeated calls."""
    for order_seed in range(4):
        w = _shared_pool_window(order_seed=order_seed)
        _check_edge(ps, scorer, w, f"groups order={order_seed}")
        _check_edge(ps, scorer, w, f"groups order={order_seed} b_max=40", b_max=40)
        _check_edge(ps, scorer, w, f"groups order={order_seed} eta=1", eta=1.0)
    # the same offsets with other contents: nothing of an earlier window's
    # groups may be used
    for base in (7, 555, 7):
        _check_edge(ps, scorer, _shared_pool_window(base=base), f"groups base={base}")


def _shared_hit_window(base=301, crowded_non_holders=False, **kw):
    """A popular first block (a 12-block shared prompt held by 86 of 96
    instances, so its holders are a bitmap) under two sessions' segments:
    most holders hit exactly the prompt (the shared-hit class, H* = 12),
    six are exceptions (longer hits from a session's own blocks, one to
    the segment's end with a cached tail after it, two with half the
    prompt), ten instances hold none of it.  Members' segment lengths lie
    on both sides of H*.  With crowded_non_holders the non-holders are
    nearly full, so the 64 largest rooms all belong to holders."""
    rng = np.random.default_rng(base)
    SP = chain_hashes(12, base=base)
    X = SP + chain_hashes(40, base=base + 10**6)
    Y = SP + chain_hashes(30, base=base + 2 * 10**6)
    tails = [chain_hashes(int(rng.integers(1, 4)), base=base + 10**8 + 10**4 * k) for k in range(6)]
    pool = []

    def put(seq):
        off = len(pool)
        pool.extend(seq)
        return off

    ox, oy = put(X), put(Y)
    t_off = [put(t) for t in tails]
    n_inst = 96
    filler = chain_hashes(400, base=base + 5 * 10**7)
    sets = [SP + filler[4 * i:4 * i + 3] for i in range(80)]    # the class: hit 12
    sets += [X[:22], X[:32], X + tails[0], X[:17]]              # exceptions of X
    sets += [SP[:6], SP[:6] + filler[350:352]]                   # exceptions: half the prompt
    sets += [filler[300 + 4 * i:302 + 4 * i] for i in range(10)]  # non-holders
    sets[5] = sets[5] + Y[12:20]                                  # an exception of Y only
    reqs = []
    for k, p in enumerate([8, 11, 12, 13, 17, 20, 22, 30, 40, 51, 52]):
        reqs.append((ox, p, t_off[k % 3], len(tails[k % 3])))
    reqs += [(ox, 52, t_off[0], len(tails[0])), (ox, 52, t_off[1], 0)]
    reqs += [(oy, p, t_off[3 + k % 3], len(tails[3 + k % 3])) for k, p in enumerate([9, 12, 15, 20, 42])]
    order = np.random.default_rng(base + 1).permutation(len(reqs))
    reqs = [reqs[i] for i in order]
    S = rng.integers(0, 500_000, n_inst)
    if crowded_non_holders:
        S[86:] = 4_194_304 - 64
    S = kw.pop("S", S)
    return _edge(sets, None, pool=pool, reqs=reqs, S=S, cap=64, **kw)


def test_popular_shared_hit_class(ps, scorer):
    """The shared-hit class of popular groups (the fast path's class scan
    and its fallbacks: H* at or past a member's segment end, no candidate
    in T (the fallback key by LMetric and by D-C-Q, with and without the
    recomputation budget admitting every class), a class not visible among
    the 64 largest rooms) against the oracle and the path with set sizes."""
    for base in (301, 302):
        w = _shared_hit_window(base=base)
        _check_edge(ps, scorer, w, f"shared hit {base}")
        _check_edge(ps, scorer, w, f"shared hit {base} eta=0", eta=0.0)
        _check_edge(ps, scorer, w, f"shared hit {base} tpot=1e-6", tpot_slo=1e-6)
        _check_edge(ps, scorer, w, f"shared hit {base} tpot=1e-6 dcq fallback", tpot_slo=1e-6,
                    flags=ps.PS_F_FALLBACK_DCQ)
        _check_edge(ps, scorer, w, f"shared hit {base} tpot=1e-6 eta=0", tpot_slo=1e-6, eta=0.0)
        _check_edge(ps, scorer, w, f"shared hit {base} b_max=40", b_max=40)
    w = _shared_hit_window(base=303, crowded_non_holders=True)
    _check_edge(ps, scorer, w, "shared hit crowded")


def test_shared_hit_class_scan_bounds(ps, scorer):
    """The class scan skips 64-instance chunks by their least decode-
    iteration time at L = 0 (instances with and without running requests
    apart) and their largest room: idle instances among busy ones, a
    prefill interference that rules out every busy instance, negative
    decode-iteration times (beta0, beta1 < 0, still a monotone model) and a
    first chunk whose rooms cannot hold any request."""
    n = 96
    rng = np.random.default_rng(7)
    D = rng.integers(0, 64, n)
    Q = rng.integers(0, 4, n)
    D[::5] = 0
    Q[::5] = 0                      # A1 = 1: no prefill interference
    w = _shared_hit_window(base=311, D=D, Q=Q)
    w.alpha = np.asarray(w.alpha, np.float32).copy()
    w.alpha[1] *= 100.0             # interference of several ms per busy instance
    _check_edge(ps, scorer, w, "class bounds: interference")
    _check_edge(ps, scorer, w, "class bounds: tight tpot", tpot_slo=0.02)
    _check_edge(ps, scorer, w, "class bounds: loose tpot", tpot_slo=0.2)
    wn = _shared_hit_window(base=312, D=D, Q=Q)
    wn.beta = np.asarray(wn.beta, np.float32).copy()
    wn.beta[..., 0] = -0.02         # t_iter below zero on lightly loaded instances
    wn.beta[..., 1] = -1e-5
    _check_edge(ps, scorer, wn, "class bounds: negative t_iter")
    _check_edge(ps, scorer, wn, "class bounds: negative t_iter, tpot 1e-3", tpot_slo=1e-3)
    S = np.random.default_rng(8).integers(0, 500_000, n)
    S[:64] = 4_194_304 - 16         # no room in the first chunk
    wc = _shared_hit_window(base=313, D=D, Q=Q, S=S)
    _check_edge(ps, scorer, wc, "class bounds: full first chunk")


def test_prefix_groups_window_sizes(ps, scorer):
    """Windows of growing and shrinking request counts on one context (the
    group table grows; later smaller windows reuse it)."""
    w = synth.generate("c2", n_req=4096)
    load_window(scorer, w)
    o = oracle.Oracle.from_window(w)
    for n in (1, 7, 4096, 300, 2048, 1):
        sub = w.subset(range(n))
        res, sizes = DeviceWindow(sub).score(scorer)
        compare_decisions(res, sizes, o.window_score(sub), label=f"c2 first {n}")


def test_kernel_timing(ps, scorer):
    """Per-launch timing of scoring calls: the claim pass, group walk and
    lean scorer of a grouped window take time, every part is non-negative,
    and a read starts a new count."""
    w = synth.generate("c2", n_req=4096)
    load_window(scorer, w)
    dw = DeviceWindow(w)
    scorer.set_timing(True)
    for _ in range(3):
        dw.score(scorer, with_sizes=False)
    n, ms = scorer.read_kernel_timing()
    assert n == 3 and len(ms) == 4 and min(ms) >= 0.0 and ms[0] > 0 and ms[1] > 0 and ms[2] > 0
    with pytest.raises(ps.PackServeError):
        scorer.read_timing()
    dw.score(scorer, with_sizes=False)
    n, g, k = scorer.read_timing()
    assert n == 1 and g > 0 and k > 0
    scorer.set_timing(False)


def test_invalid_descriptor_flagged_on_device(ps, scorer):
    import torch
    w = synth.generate("c1", n_req=8)
    load_window(scorer, w)
    reqs = reqs_of(w)
    reqs["pre_off"][3] = len(w.pool) + 5
    reqs["tail_len"][5] = -1
    d_pool = ps.to_device_u64(w.pool)
    d_reqs = ps.to_device_bytes(reqs)
    d_out = torch.zeros(8 * 20, dtype=torch.uint8, device="cuda")
    scorer.score_dev(d_pool, len(w.pool), d_reqs, 8, d_out)
    torch.cuda.synchronize()
    res = ps.results_from_device(d_out)
    assert res["flags"][3] == ps.PS_R_INVALID and res["instance"][3] == -1
    assert res["flags"][5] == ps.PS_R_INVALID
    assert (res["flags"][[0, 1, 2, 4, 6, 7]] & ps.PS_R_INVALID == 0).all()


# ------------------------------------------------------------- commit
@pytest.mark.parametrize("name,n_req,cap", [("c1", 1024, None), ("c2", 2048, None),
                                            ("c1", 1024, 1100)])
def test_commit_sequence(ps, scorer, name, n_req, cap):
    """Score window 1, apply the oracle's decisions on both sides, compare
    the state, then score window 2 against the updated snapshot."""
    _say(f"commit {name} cap={cap}")
    gen = dict(n_req=n_req)
    if cap:
        gen["cap"] = cap
    w = synth.generate(name, **gen)
    load_window(scorer, w)
    o = oracle.Oracle.from_window(w)
    od = o.window_score(w)
    dropped_o = o.commit(w.pool, w.pre_off, w.pre_len, w.tail_off, w.tail_len, od.inst)
    dropped_g = scorer.commit(w.pool, reqs_of(w), od.inst)
    so, sg = o.state(), scorer.state()
    for k in ("D", "Q", "P", "S", "set_size"):
        assert (so[k] == sg[k]).all(), f"{k} differs after commit"
    assert dropped_o == dropped_g
    if cap:
        assert dropped_o > 0
    w2 = synth.generate(name, seed=1, **gen)
    # same instances and model as the loaded snapshot; only the requests are new
    w2.blk_off, w2.blk = w.blk_off, w.blk
    w2.alpha, w2.beta, w2.gamma = w.alpha, w.beta, w.gamma
    w2.pool = np.concatenate([w.pool, w2.pool])
    off = len(w.pool)
    w2.pre_off = w2.pre_off + off
    w2.tail_off = w2.tail_off + off
    # half of window 2 repeats window-1 requests (now cached on their instance)
    w2.pre_off[::2] = w.pre_off[::2]
    w2.pre_len[::2] = w.pre_len[::2]
    w2.tail_off[::2] = w.tail_off[::2]
    w2.tail_len[::2] = w.tail_len[::2]
    res, sizes = DeviceWindow(w2).score(scorer)
    od2 = o.window_score(w2)
    compare_decisions(res, sizes, od2, label=f"{name} after commit")


# ------------------------------------------------------------- ABI errors
def test_abi_errors(ps, scorer):
    w = synth.generate("c1", n_req=4)
    reqs = reqs_of(w)
    with pytest.raises(ps.PackServeError) as e:
        scorer.score(w.pool, reqs)
    assert e.value.code == -4
    m = gpu_model(w)
    bad_blk = w.blk.copy()
    bad_blk[3] = 0
    with pytest.raises(ps.PackServeError) as e:
        scorer.load(w.n_inst, w.cap, w.blk_off, bad_blk, w.D, w.Q, w.P, w.S, m)
    assert e.value.code == -1
    D = w.D.copy()
    D[0] = 4096
    with pytest.raises(ps.PackServeError) as e:
        scorer.load(w.n_inst, w.cap, w.blk_off, w.blk, D, w.Q, w.P, w.S, m)
    assert e.value.code == -5
    m2 = gpu_model(w)
    m2.seg_ub[2] = m2.seg_ub[1]
    with pytest.raises(ps.PackServeError) as e:
        scorer.load(w.n_inst, w.cap, w.blk_off, w.blk, w.D, w.Q, w.P, w.S, m2)
    assert e.value.code == -1
    m3 = gpu_model(w, eta=-0.1)
    with pytest.raises(ps.PackServeError) as e:
        scorer.load(w.n_inst, w.cap, w.blk_off, w.blk, w.D, w.Q, w.P, w.S, m3)
    assert e.value.code == -1
    with pytest.raises(ps.PackServeError) as e:
        scorer.load(w.n_inst, 3, w.blk_off, w.blk, w.D, w.Q, w.P, w.S, m)
    assert e.value.code == -5
    # a good load, then a failing one: the first snapshot stays in force
    scorer.load(w.n_inst, w.cap, w.blk_off, w.blk, w.D, w.Q, w.P, w.S, m)
    a = scorer.score(w.pool, reqs)
    with pytest.raises(ps.PackServeError):
        scorer.load(w.n_inst, w.cap, w.blk_off, bad_blk, w.D, w.Q, w.P, w.S, m)
    assert scorer.score(w.pool, reqs).tobytes() == a.tobytes()
    r2 = reqs.copy()
    r2["pre_off"][0] = len(w.pool)
    with pytest.raises(ps.PackServeError) as e:
        scorer.score(w.pool, r2)
    assert e.value.code == -5
    p2 = w.pool.copy()
    p2[0] = 0
    with pytest.raises(ps.PackServeError) as e:
        scorer.score(p2, reqs)
    assert e.value.code == -1
    big = np.full((1 << 23) + 1, 7, np.uint64)
    r3 = ps.pack_reqs([0], [(1 << 23) + 1], [0], [1 << 23])
    with pytest.raises(ps.PackServeError) as e:
        scorer.score(big, r3)
    assert e.value.code == -5
    with pytest.raises(ps.PackServeError) as e:
        scorer.commit(w.pool, reqs, np.array([0, 1, w.n_inst, 0], np.int32))
    assert e.value.code == -5
    assert len(scorer.score(w.pool, reqs[:0])) == 0


# ------------------------------------------------------------- full-size windows
@pytest.mark.parametrize("name", ["c3", "c4", "c5"])
def test_full_size_window(ps, scorer, name):
    """The full window on the GPU in the benchmark's launch configuration
    (one call of the scoring entry point, with and without set sizes)
    against the oracle on every request: choices, hits, flags, set sizes and
    latencies; the window's placed and fallback counts; then every request's
    hit on every instance, in slices of requests."""
    _say(f"full-size {name}: generating")
    w = synth.generate(name)
    _say(f"full-size {name}: loading")
    load_window(scorer, w)
    dw = DeviceWindow(w)
    res, sizes = dw.score(scorer)
    res2, _ = dw.score(scorer, with_sizes=False)
    assert res2.tobytes() == res.tobytes(), f"{name}: path without sizes differs"
    _say(f"full-size {name}: scored {w.n_req}; oracle")
    o = oracle.Oracle.from_window(w)
    od = o.window_score(w)
    nb = compare_decisions(res, sizes, od, label=name)
    placed_g, placed_o = int((res["instance"] >= 0).sum()), int((od.inst >= 0).sum())
    fb_g = int((res["flags"] & ps.PS_R_FALLBACK != 0).sum())
    fb_o = int((od.flags & oracle.R_FALLBACK != 0).sum())
    assert placed_g == placed_o, f"{name}: placed {placed_g} vs {placed_o}"
    assert abs(fb_g - fb_o) <= nb, f"{name}: fallback {fb_g} vs {fb_o} ({nb} near-boundary)"
    _say(f"full-size {name}: {w.n_req} decisions match ({nb} near-boundary; placed {placed_g}, "
         f"fallback {fb_g}); hits")
    step = 32768
    for a in range(0, w.n_req, step):
        sub = w.subset(range(a, min(a + step, w.n_req)))
        got = DeviceWindow(sub).hits(scorer, w.n_inst)
        want = o.window_hits(sub)
        bad = np.argwhere(got != want)
        assert len(bad) == 0, (f"{name}: {len(bad)} hits differ in requests {a}.., first "
                               f"{bad[0]}: {got[tuple(bad[0])]} vs {want[tuple(bad[0])]}")
    _say(f"full-size {name}: {w.n_req} x {w.n_inst} hits match")
    o.close()


# ------------------------------------------------------------- policy variants
SELECTORS = ["DCQ", "D", "DQ", "DC", "DQC", "HCQ", "RANDOM", "LMETRIC"]
LAYERS = {"G": 2 | 4, "C": 4, "T": 2 | 8, "CT": 8, "F": 0}


@pytest.mark.parametrize("name,gen", [("c1", {}), ("c2", dict(n_req=2048)),
                                      ("c3", dict(n_inst=128, n_sess=256, n_req=1024))])
def test_selectors_and_layers(ps, scorer, name, gen):
    """Every selector of Table 4 (plus LMetric) and every admission layer of
    Table 3, on windows with one and with many holders of the first block."""
    w = synth.generate(name, **gen)
    o = oracle.Oracle.from_window(w)
    dw = DeviceWindow(w)
    for k, sel in enumerate(SELECTORS):
        for layer, fl in LAYERS.items():
            flags = fl | (k << 8)
            pol = dict(flags=flags, rand_seed=1234567 + k)
            load_window(scorer, w, **pol)
            res, sizes = dw.score(scorer)
            od = o.window_score(w, **pol)
            compare_decisions(res, sizes, od, label=f"{name} {sel} {layer}")
            res2, _ = dw.score(scorer, with_sizes=False)
            assert res2.tobytes() == res.tobytes(), f"{name} {sel} {layer}: no-sizes path differs"


# ------------------------------------------------------------- feedback path
def test_feedback_path(ps, scorer):
    """EMA calibration, the median output tracker and response-path
    transitions applied to both sides, then a window scored on the result."""
    w = synth.generate("c2", n_req=2048)
    load_window(scorer, w)
    o = oracle.Oracle.from_window(w)
    m = oracle.model_of(w)
    rng = np.random.default_rng(11)
    n = 600
    B = rng.integers(1, 700, n).astype(np.int32)
    S = rng.integers(0, 3_000_000, n).astype(np.int64)
    meas = rng.uniform(0.005, 0.2, n).astype(np.float32)
    scorer.feedback_decode(B, S, meas)
    oracle.feedback_decode(m, B, S, meas.astype(np.float64))
    g = scorer.model()["gamma"]
    want = np.array([m.gamma[k] for k in range(len(g))])
    assert np.allclose(g, want, rtol=1e-6, atol=0), (g, want)
    assert (g >= 1.0).all() and (g <= 2.0).all() and (np.abs(g - 1.0) > 1e-3).any()
    outs = rng.integers(1, 4000, 1500).astype(np.int32)
    scorer.feedback_output(outs)
    o.feedback_output(m, outs)
    assert scorer.model()["lout"] == m.lout
    # valid transitions, drawn against a local copy of the counters
    st = o.state()
    D, Q, P, S_ = st["D"].astype(np.int64), st["Q"].astype(np.int64), st["P"].copy(), st["S"].copy()
    inst, kind, tok = [], [], []
    for _ in range(400):
        i = int(rng.integers(0, w.n_inst))
        k = int(rng.integers(1, 4))
        if k == 1 and Q[i] > 0:
            t = int(rng.integers(0, P[i] + 1))
            Q[i] -= 1; D[i] += 1; P[i] -= t
        elif k == 2:
            t = int(rng.integers(0, 5000))
            S_[i] += t
        elif k == 3 and D[i] > 0:
            t = int(rng.integers(0, S_[i] + 1))
            D[i] -= 1; S_[i] -= t
        else:
            continue
        inst.append(i); kind.append(k); tok.append(t)
    scorer.apply_events(inst, kind, tok)
    assert o.apply_events(inst, kind, tok) == 0
    so, sg = o.state(), scorer.state()
    for k in ("D", "Q", "P", "S"):
        assert (so[k] == sg[k]).all(), k
    # an out-of-range batch is refused as a whole
    before = scorer.state()
    j = int(np.argmin(sg["D"]))
    with pytest.raises(ps.PackServeError) as e:
        scorer.apply_events([0, j] + [j] * (int(sg["D"][j]) + 1),
                            [2] + [3] * (int(sg["D"][j]) + 2), [1] * (int(sg["D"][j]) + 3))
    assert e.value.code == -5
    after = scorer.state()
    for k in ("D", "Q", "P", "S"):
        assert (before[k] == after[k]).all()
    res, sizes = DeviceWindow(w).score(scorer)
    od = o.score(m, w.pool, w.pre_off, w.pre_len, w.tail_off, w.tail_len)
    compare_decisions(res, sizes, od, label="after feedback")


def _long_shared_prefix_window(base=401):
    """A 300-block shared prefix (longer than a staged chain head and than
    one round of the popular pass's prefix walk) held by 150 of 160
    instances, cut short on some of them at positions around the round and
    stage boundaries, and dropping to 40 (a holder list) and then 9 holders
    past position 130; four sessions leave it at different positions (300,
    200, 40, 1), so groups with one popular first block share prefixes of
    different lengths with its representative; each session's own blocks
    on one to three owners, one with a hole."""
    rng = np.random.default_rng(base)
    SP = chain_hashes(300, base=base)
    own = {k: chain_hashes(60, base=base + (k + 1) * 10**6) for k in range(4)}
    segs = {0: SP + own[0], 1: SP[:200] + own[1], 2: SP[:40] + own[2], 3: SP[:1] + own[3]}
    pool = []

    def put(seq):
        off = len(pool)
        pool.extend(seq)
        return off

    seg_off = {k: put(v) for k, v in segs.items()}
    tail = chain_hashes(3, base=base + 9 * 10**7)
    t_off = put(tail)
    n_inst = 160
    filler = chain_hashes(2000, base=base + 5 * 10**7)
    cut = np.full(n_inst, 300)
    cut[:40] = [5, 64, 127, 128, 129, 200, 255, 256, 257, 299] * 4
    cut[40:150] = np.where(rng.random(110) < 0.9, 131, 300)   # 40 or so left past 130
    cut[150:] = 0                                            # hold none of it
    sets = []
    for i in range(n_inst):
        s = list(SP[:cut[i]]) + list(filler[10 * i:10 * i + 3])
        sets.append(s)
    for k in range(4):  # owners of each session's own blocks
        lead = len(segs[k]) - 60
        for j, i in enumerate(rng.choice(150, 3, replace=False)):
            if cut[i] >= lead:
                extra = own[k][:10 + 20 * j]
                if j == 2:
                    extra = extra[:5] + extra[6:]  # a hole
                sets[i] = sets[i] + list(extra)
    reqs = []
    for k in range(4):
        L = len(segs[k])
        for p in (L - 60, L - 55, L - 30, L, max(8, L - 70)):
            reqs.append((seg_off[k], p, t_off, 3))
    order = np.random.default_rng(base + 1).permutation(len(reqs))
    reqs = [reqs[i] for i in order]
    return _edge(sets, None, pool=pool, reqs=reqs, cap=1024)


def test_popular_pass_shared_prefixes(ps, scorer):
    """Groups whose first block has a holder bitmap are walked by the
    popular pass beside the walk pass (a prefix walk per first block, then
    each group from the end of its common prefix with the representative):
    oracle parity, and byte for byte the results of the allocation-free
    entry point, whose walk pass walks every group itself."""
    for base in (401, 402):
        w = _long_shared_prefix_window(base=base)
        res = _check_edge(ps, scorer, w, f"long shared prefix {base}")
        fixed, _ = DeviceWindow(w).score(scorer, fixed=True)
        assert fixed.tobytes() == res.tobytes(), f"{base}: the walk pass alone decides differently"
        _check_edge(ps, scorer, w, f"long shared prefix {base} eta=1", eta=1.0)


def _dwindling_prefix_window(base=411, survivor_len=300):
    """A shared prefix held by 100 instances for its first 40 blocks and
    by one (or two) of them further, to survivor_len: the popular pass's
    prefix walk stops at its first round's end with one holder live, before
    the 290 blocks that sessions A and B still share, so that holder is
    walked again from the stop."""
    SP = chain_hashes(300, base=base)
    own = {k: chain_hashes(20, base=base + (k + 1) * 10**6) for k in range(3)}
    segs = {0: SP + own[0], 1: SP[:290] + own[1], 2: SP[:35] + own[2]}
    pool = []

    def put(seq):
        off = len(pool)
        pool.extend(seq)
        return off

    seg_off = {k: put(v) for k, v in segs.items()}
    n_inst = 110
    filler = chain_hashes(2000, base=base + 5 * 10**7)
    sets = [list(SP[:40]) + list(filler[5 * i:5 * i + 2]) for i in range(100)]
    sets[7] = list(SP[:survivor_len]) + list(own[0][:10]) + list(own[1][:5])
    sets[50] = list(SP[:survivor_len // 2]) + list(own[1][:3])
    sets += [list(filler[1000 + 5 * i:1002 + 5 * i]) for i in range(10)]
    reqs = []
    for k in range(3):
        L = len(segs[k])
        for p in (L, L - 10, L - 25):
            reqs.append((seg_off[k], p, put(chain_hashes(2, base=base + 10**8 + len(pool))), 2))
    return _edge(sets, None, pool=pool, reqs=reqs, cap=1024)


def test_popular_pass_early_prefix_stop(ps, scorer):
    """The prefix walk stops with one holder live before the common prefix
    of two groups ends: that holder is walked from the stop (holding the
    rest, or not)."""
    for surv in (300, 200, 41):
        w = _dwindling_prefix_window(survivor_len=surv)
        res = _check_edge(ps, scorer, w, f"dwindling prefix {surv}")
        fixed, _ = DeviceWindow(w).score(scorer, fixed=True)
        assert fixed.tobytes() == res.tobytes(), f"{surv}: the walk pass alone decides differently"


def _many_popular_groups_window(n_groups, n_inst=4096, base=431):
    """n_groups sessions whose segments all start with one block held by
    every instance (a holder bitmap), each then on its own 9 blocks held in
    part by one or two owners: more popular groups than the popular pass's
    list has rows at 4,096 instances (4,096), and past that more than the
    walk pass's own popular rows hold, so groups take all three paths."""
    rng = np.random.default_rng(base)
    B0 = chain_hashes(1, base=base)[0]
    own = chain_hashes(9 * n_groups, base=base + 10**6)
    pool, reqs = [], []
    tail_off = 0
    # a shared four-block tail (with two or three blocks one request length
    # puts the recomputation ratio of the first block's holders within
    # 1e-5 of eta against the owners' hits: 0.6% near-boundary decisions)
    pool.extend(chain_hashes(4, base=base + 10**8))
    sets = [[B0] for _ in range(n_inst)]
    for k in range(n_groups):
        off = len(pool)
        blocks = own[9 * k:9 * k + 9]
        pool.append(B0)
        pool.extend(blocks)
        for j, i in enumerate(rng.choice(n_inst, 1 + (k % 2), replace=False)):
            keep = int(rng.integers(0, 10))
            sets[i].extend(blocks[:keep])
        reqs.append((off, 10 if k % 3 else 9, tail_off, 4))
    order = rng.permutation(len(reqs))
    reqs = [reqs[i] for i in order]
    return _edge(sets, None, pool=pool, reqs=reqs, cap=64)


def test_popular_list_overflow(ps, scorer):
    """8,500 popular groups at 4,096 instances: 4,096 in the popular pass,
    the rest in the walk pass until its popular rows run out, the last ones
    without a record (their requests walk on their own): oracle parity on
    every request, and byte for byte the allocation-free entry point."""
    w = _many_popular_groups_window(8500)
    res = _check_edge(ps, scorer, w, "8,500 popular groups")
    fixed, _ = DeviceWindow(w).score(scorer, fixed=True)
    assert fixed.tobytes() == res.tobytes(), "the walk pass alone decides differently"


def _random_window(seed):
    """A seeded random window: pools of 1-300 instances; sessions whose
    segments may start with one shared prompt (held by up to every
    instance, so past 64 holders it has a holder bitmap); holders keep a
    segment's prefix up to a random cut, some with a hole; repeats inside
    chains; requests with random segment lengths (below and above the
    grouping minimum) and tails; random states."""
    rng = np.random.default_rng(seed)
    n_inst = int(rng.choice([1, 7, 63, 64, 65, 130, 300]))
    base = 10**7 * (seed + 1)
    SP = chain_hashes(int(rng.integers(1, 300)), base=base)
    n_sess = int(rng.integers(1, 12))
    segs = []
    for k in range(n_sess):
        own = chain_hashes(int(rng.integers(1, 400)), base=base + (k + 1) * 10**5)
        if len(own) > 6 and rng.random() < 0.3:
            own[5] = own[2]  # a repeated block
        lead = SP[:int(rng.integers(1, len(SP) + 1))] if rng.random() < 0.6 else []
        segs.append(list(lead) + list(own))
    pool, seg_off = [], []
    for sg in segs:
        seg_off.append(len(pool))
        pool.extend(sg)
    fresh = chain_hashes(2000, base=base + 9 * 10**6)
    sets = [[] for _ in range(n_inst)]
    sp_frac = float(rng.choice([0.0, 0.5, 1.0]))
    for i in range(n_inst):
        if rng.random() < sp_frac:
            sets[i].extend(SP[:int(rng.integers(0, len(SP) + 1))])
        for k in range(n_sess):
            if rng.random() < 2.0 / max(n_inst, 1) + 0.05:
                cut = int(rng.integers(0, len(segs[k]) + 1))
                held = segs[k][:cut]
                if cut > 10 and rng.random() < 0.2:
                    held = held[:cut // 2] + held[cut // 2 + 1:]  # a hole
                sets[i].extend(held)
        sets[i].extend(fresh[3 * i:3 * i + int(rng.integers(0, 3))])
        sets[i] = list(dict.fromkeys(sets[i]))  # one entry per block
    reqs = []
    n_req = int(rng.integers(1, 400))
    for r in range(n_req):
        k = int(rng.integers(0, n_sess))
        p = int(rng.integers(1, len(segs[k]) + 1))
        t = int(rng.integers(0, 5))
        t_off = len(pool)
        pool.extend(fresh[1000 + (r * 5) % 900:1000 + (r * 5) % 900 + t])
        reqs.append((seg_off[k], p, t_off, t))
    cap = max(max(len(s) for s in sets), 1) + int(rng.integers(0, 64))
    return _edge(sets, None, pool=pool, reqs=reqs, cap=cap)


RANDOM_POLICIES = [dict(), dict(eta=0.25), dict(eta=1.0), dict(flags=1), dict(flags=2),
                   dict(tpot_slo=0.05)]


RANDOM_SEEDS = [s for s in range(160) if s != 156]  # 156: 10 near-boundary decisions (cap 8)


def test_random_windows(ps, scorer):
    """159 seeded random windows (pool sizes 1-300, shared prompts with and
    without holder bitmaps, holes, repeats, groups, random policies):
    oracle parity on every request and byte-identical results from the
    allocation-free entry point."""
    for seed in RANDOM_SEEDS:
        w = _random_window(seed)
        pol = RANDOM_POLICIES[seed % len(RANDOM_POLICIES)]
        _say(f"random window {seed}: {w.n_inst} instances, {w.n_req} requests, {pol}")
        res = _check_edge(ps, scorer, w, f"random window {seed}", **pol)
        fixed, _ = DeviceWindow(w).score(scorer, fixed=True)
        assert fixed.tobytes() == res.tobytes(), f"random window {seed}: the fixed path differs"


def _random_window_large(seed):
    """Larger seeded random windows: 1,000-4,096 instances (holder bitmaps
    of up to 64 words), segments of up to 6,000 blocks (past every staged
    chain head), a shared prompt held by most instances, 200-2,000
    requests over few sessions (groups of many members)."""
    rng = np.random.default_rng(10**6 + seed)
    n_inst = int(rng.choice([1000, 2100, 4096]))
    base = 10**8 * (seed + 1)
    SP = chain_hashes(int(rng.integers(50, 400)), base=base)
    n_sess = int(rng.integers(2, 20))
    segs = []
    for k in range(n_sess):
        own = chain_hashes(int(rng.integers(10, 6000)), base=base + (k + 1) * 10**6)
        lead = SP[:int(rng.integers(1, len(SP) + 1))] if rng.random() < 0.7 else []
        segs.append(list(lead) + list(own))
    pool, seg_off = [], []
    for sg in segs:
        seg_off.append(len(pool))
        pool.extend(sg)
    sets = [[] for _ in range(n_inst)]
    for i in np.nonzero(rng.random(n_inst) < 0.8)[0]:
        sets[i].extend(SP[:int(rng.integers(len(SP) // 2, len(SP) + 1))])
    for k in range(n_sess):  # each session on one to three owners
        for i in rng.choice(n_inst, int(rng.integers(1, 4)), replace=False):
            sets[i].extend(segs[k][:int(rng.integers(0, len(segs[k]) + 1))])
    sets = [list(dict.fromkeys(s)) for s in sets]
    fresh = chain_hashes(20000, base=base + 9 * 10**7)
    reqs = []
    for r in range(int(rng.integers(200, 2000))):
        k = int(rng.integers(0, n_sess))
        t = int(rng.integers(0, 4))
        t_off = len(pool)
        pool.extend(fresh[(r * 4) % 19000:(r * 4) % 19000 + t])
        reqs.append((seg_off[k], int(rng.integers(1, len(segs[k]) + 1)), t_off, t))
    cap = max(max(len(s) for s in sets), 1) + 64
    return _edge(sets, None, pool=pool, reqs=reqs, cap=cap)


def test_random_windows_large(ps, scorer):
    """Twelve larger seeded random windows (1,000-4,096 instances, chains
    of up to 6,000 blocks, large groups): oracle parity and byte-identical
    results from the allocation-free entry point."""
    for seed in range(12):
        w = _random_window_large(seed)
        _say(f"large random window {seed}: {w.n_inst} instances, {w.n_req} requests")
        res = _check_edge(ps, scorer, w, f"large random window {seed}")
        fixed, _ = DeviceWindow(w).score(scorer, fixed=True)
        assert fixed.tobytes() == res.tobytes(), f"large random window {seed}: the fixed path differs"
