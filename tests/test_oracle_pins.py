"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself or with a retyped copy of its
formulas: the expected values are hand-computed (tests/golden), closed forms
and special cases the paper states, brute force at the token level, and
invariants of Algorithm 1.
"""
import hashlib
import json
import os

import numpy as np
import pytest

import oracle
import synth
from tests.tinywin import chain_hashes, make_window

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")
FLAGS = dict(TTFT_ADMIT=oracle.F_TTFT_ADMIT, NO_KVC_FILTER=oracle.F_NO_KVC_FILTER,
             NO_TPOT_FILTER=oracle.F_NO_TPOT_FILTER)
RFLAGS = dict(REJECT=oracle.R_REJECT, FALLBACK=oracle.R_FALLBACK, TTFT_MISS=oracle.R_TTFT_MISS)


def _flagbits(v, table):
    if isinstance(v, list):
        out = 0
        for name in v:
            out |= table[name]
        return out
    return int(v)


def _worked_window(g, b_max, eta, tau, flags):
    L = g["chain_blocks"]
    ch = chain_hashes(L)
    sets = []
    for inst in g["instances"]:
        h = inst["hit"]
        # instance 4 (hit 0) holds every block but the first one
        sets.append(ch[:h] if h > 0 else ch[1:])
    inst = g["instances"]
    return make_window(
        sets, [ch], D=[x["D"] for x in inst], Q=[x["Q"] for x in inst],
        P=[x["P"] for x in inst], S=[x["S"] for x in inst], alpha=g["alpha"],
        seg_ub=g["seg_ub"], beta=g["beta"], gamma=g["gamma"], eta=eta, tpot_slo=tau,
        ttft_floor=g["ttft_floor"], lout=g["lout"], block_tokens=g["block_tokens"],
        b_max=b_max, kv_cap_tokens=g["kv_cap"], flags=flags, cap=16)


def _decide(win, **policy):
    o = oracle.Oracle.from_window(win)
    try:
        return o.window_score(win, nthreads=1, **policy)
    finally:
        o.close()


@pytest.fixture(scope="module")
def gold():
    with open(GOLD) as f:
        return json.load(f)


# -- hand-worked example (Algorithm 1, Eqs. 7-10) ---------------------------

def test_worked_example_cases(gold):
    for case in gold["cases"]:
        fl = _flagbits(case["flags"], FLAGS)
        win = _worked_window(gold, case["b_max"], case["eta"], case["tau"], fl)
        d = _decide(win)
        assert d.inst[0] == case["inst"], case["name"]
        assert d.hit[0] == case["hit"], case["name"]
        assert d.flags[0] == _flagbits(case["rflags"], RFLAGS), case["name"]
        if case["inst"] >= 0:
            assert d.ttft[0] == pytest.approx(case["ttft"], rel=1e-6), case["name"]
            assert d.tpot[0] == pytest.approx(case["tpot"], rel=1e-6), case["name"]
        if case["sizes"] is not None:
            assert list(d.sizes[0]) == case["sizes"], case["name"]
        if case.get("near_boundary"):
            assert d.nb[0] & oracle.NB_RHO, case["name"]
        else:
            assert d.nb[0] & oracle.NB_DECISION == 0, case["name"]


def test_worked_example_per_instance_latencies(gold):
    """Each instance alone, filters off: the decision exposes its TTFT/TPOT."""
    per = gold["derived"]["per_instance"]
    for i, inst in enumerate(gold["instances"]):
        g1 = dict(gold)
        g1["instances"] = [inst]
        win = _worked_window(g1, 1000, 0.5, 1.0, oracle.F_NO_KVC_FILTER | oracle.F_NO_TPOT_FILTER)
        d = _decide(win)
        assert d.inst[0] == 0 and d.hit[0] == inst["hit"]
        assert d.tpot[0] == pytest.approx(per[i]["tpot"], rel=1e-9)
        assert d.ttft[0] == pytest.approx(per[i]["ttft"], rel=1e-9)


# -- special cases the paper states -----------------------------------------

SIMPLE_ALPHA = [0.02, 1e-3, 1e-6, 1e-6, 1e-5, 2e-9]


def _one_inst(hit, L=8, D=0, Q=0, P=0, S=0, alpha=SIMPLE_ALPHA, seg_ub=(64,),
              beta=((0.01, 1e-4, 1e-8),), gamma=(1.0,), **pol):
    ch = chain_hashes(L)
    pol.setdefault("tpot_slo", 10.0)
    pol.setdefault("b_max", 10_000)
    pol.setdefault("kv_cap_tokens", 10**9)
    return make_window([ch[:hit]], [ch], [D], [Q], [P], [S], alpha, seg_ub, beta, gamma,
                       cap=max(hit, 1), **pol)


def test_interference_term_dropped_when_idle():
    """Eq. 10: the prefill-interference term is omitted when A_i = 0."""
    a, b = SIMPLE_ALPHA, (0.01, 1e-4, 1e-8)
    L, hit, S = 8 * 16, 3, 5000
    n, c = L - hit * 16, hit * 16
    tpf = a[0] + a[1] * n + a[2] * n * c + a[3] * n * n + a[4] * c + a[5] * c * c
    idle = _decide(_one_inst(hit, S=S))
    assert idle.tpot[0] == pytest.approx(b[0] + b[1] * 1 + b[2] * (S + L), rel=1e-12)
    busy = _decide(_one_inst(hit, D=1, S=S))
    assert busy.tpot[0] == pytest.approx(b[0] + b[1] * 2 + b[2] * (S + L) + tpf / 556.0, rel=1e-12)


def test_fully_cached_prefill_cost():
    """n = 0: T_pf(0, L) = a0 + a4 L + a5 L^2; TTFT adds a0 Q + a1 P."""
    a = SIMPLE_ALPHA
    L = 8 * 16
    d = _decide(_one_inst(8, Q=2, P=300, D=1))
    assert d.hit[0] == 8
    tpf = a[0] + a[4] * L + a[5] * L * L
    assert d.ttft[0] == pytest.approx(tpf + a[0] * 2 + a[1] * 300, rel=1e-12)


def test_single_segment_reduces_to_eq8():
    """One segment with gamma = 1: the decode term is Eq. 8 itself, and the
    EMA factor scales only that term (Sec. 5.3)."""
    beta = (0.004, 3e-4, 2e-8)
    d1 = _decide(_one_inst(2, D=0, Q=0, S=1234, seg_ub=(8,), beta=(beta,), gamma=(1.0,)))
    L = 128
    assert d1.tpot[0] == pytest.approx(beta[0] + beta[1] * 1 + beta[2] * (1234 + L), rel=1e-12)
    d2 = _decide(_one_inst(2, D=0, Q=0, S=1234, seg_ub=(8,), beta=(beta,), gamma=(1.5,)))
    assert d2.tpot[0] == pytest.approx(1.5 * d1.tpot[0], rel=1e-12)


def test_segment_bounds_inclusive_and_last_segment():
    """B+ equal to a bound uses that segment; past the last bound, the last."""
    beta = ((1.0, 0, 0), (2.0, 0, 0), (3.0, 0, 0))
    ub = (4, 8, 16)
    for active, want in [(3, 1.0), (4, 2.0), (7, 2.0), (8, 3.0), (15, 3.0), (40, 3.0)]:
        d = _decide(_one_inst(0, D=active, Q=0, alpha=[0] * 6, seg_ub=ub, beta=beta,
                              gamma=(1, 1, 1), tpot_slo=100.0))
        assert d.tpot[0] == pytest.approx(want), active


def _multi(hits, L=8, D=None, Q=None, P=None, S=None, alpha=SIMPLE_ALPHA, **pol):
    ch = chain_hashes(L)
    n = len(hits)
    D = D if D is not None else [0] * n
    Q = Q if Q is not None else [0] * n
    P = P if P is not None else [0] * n
    S = S if S is not None else [0] * n
    pol.setdefault("tpot_slo", 10.0)
    pol.setdefault("b_max", 10_000)
    pol.setdefault("kv_cap_tokens", 10**9)
    sets = [ch[:h] for h in hits]
    return make_window(sets, [ch], D, Q, P, S, alpha, (10_000,), ((0.001, 0, 0),), (1.0,),
                       cap=L, **pol)


def test_zero_cache_benefit_keeps_all():
    """Sec. 6.1: if Z_r = 0 all capacity-eligible candidates remain (here
    T_pf = a0 + a2 N C, so T_pf(L,0) = T_pf(0,L)), even with eta = 0."""
    alpha = [0.02, 0, 1e-6, 0, 0, 0]
    d = _decide(_multi([0, 3, 5, 8], alpha=alpha, eta=0.0))
    assert list(d.sizes[0]) == [4, 4, 4]
    assert d.nb[0] & oracle.NB_Z


def test_eta_zero_keeps_minimum_cost_only():
    """Sec. 6.1: eta = 0 retains only minimum-cost candidates."""
    d = _decide(_multi([2, 6, 6, 5, 0], eta=0.0))
    assert list(d.sizes[0][:2]) == [5, 2]
    assert d.hit[0] == 6 and d.inst[0] == 1


def test_recompute_cost_clamp_binds():
    """W is the nonnegative penalty (Sec. 6.1).  With T_pf = N^2/32 + C
    (alpha3 = 1/32, alpha4 = 1) and L = 128: T_pf(n, L-n) - T_pf(0, L) =
    n (n/32 - 1), so hits 8, 7, 4, 0 give raw penalties 0, -8, 64, 384 and
    W = 0, 0, 64, 384; Z = 384, rho = 0, 0, 1/6, 1.  With eta = 0.17 the
    instance with hit 4 is admissible and, being the only one decoding,
    wins; without the clamp its rho would be 72/384 > 0.17."""
    alpha = [0, 0, 0, 1.0 / 32, 1.0, 0]
    d = _decide(_multi([8, 7, 4, 0], alpha=alpha, eta=0.17, D=[0, 0, 5, 0]))
    assert list(d.sizes[0][:2]) == [4, 3]
    assert d.inst[0] == 2 and d.hit[0] == 4


def test_rho_boundary_is_inclusive():
    """Alg. 1 keeps rho <= eta.  With T_pf = N, rho = (n_i - n_min) / L is
    exact in binary: hits 8 and 4 of 8 blocks give rho = 0.5."""
    alpha = [0, 1.0, 0, 0, 0, 0]
    d = _decide(_multi([8, 4], alpha=alpha, eta=0.5, D=[0, 5]))
    assert list(d.sizes[0][:2]) == [2, 2] and d.inst[0] == 1
    d = _decide(_multi([8, 4], alpha=alpha, eta=0.49, D=[0, 5]))
    assert list(d.sizes[0][:2]) == [2, 1] and d.inst[0] == 0


def test_tpot_boundary_is_strict():
    """Alg. 1 keeps predicted TPOT < tau (strict): a TPOT equal to tau fails."""
    w = _one_inst(0, alpha=[0] * 6, beta=((0.5, 0, 0),), tpot_slo=0.5)
    d = _decide(w)
    assert d.flags[0] & oracle.R_FALLBACK and d.sizes[0][2] == 0
    d = _decide(w, tpot_slo=0.5000001)
    assert not d.flags[0] & oracle.R_FALLBACK and d.sizes[0][2] == 1


def test_ttft_admission_boundary_is_inclusive():
    """With TTFT admission on, TTFT <= budget passes (budget = max(floor,
    T_pf(L,0)), Sec. 8.1).  T_pf = 1 + N makes TTFT = 1 + n exactly."""
    alpha = [1.0, 1.0, 0, 0, 0, 0]
    # L = 16 tokens, hit 0: TTFT = 17 = T_pf(L,0) = budget -> admitted
    w = _one_inst(0, L=1, alpha=alpha, beta=((0.001, 0, 0),), flags=oracle.F_TTFT_ADMIT,
                  ttft_floor=2.0)
    d = _decide(w)
    assert d.sizes[0][2] == 1 and d.ttft[0] == 17.0 and not d.flags[0] & oracle.R_TTFT_MISS
    # one queued request adds a0 = 1 second of queueing: 18 > 17 -> fallback
    w = _one_inst(0, L=1, Q=1, alpha=alpha, beta=((0.001, 0, 0),), flags=oracle.F_TTFT_ADMIT)
    d = _decide(w)
    assert d.sizes[0][2] == 0 and d.flags[0] & oracle.R_FALLBACK and d.flags[0] & oracle.R_TTFT_MISS


def test_capacity_bounds_inclusive():
    """A_i + 1 <= B_max and S_i + L_r <= M_KV (reading of CapacityCandidates
    from the batch bound of Sec. 3)."""
    L = 128
    d = _decide(_multi([0, 0, 0, 0], D=[6, 7, 0, 0], Q=[1, 1, 0, 0], S=[0, 0, 1000 - L, 1001 - L],
                       b_max=8, kv_cap_tokens=1000))
    # instance 0: A+1 = 8 ok; 1: 9 > 8; 2: S+L = 1000 ok; 3: 1001 > 1000
    assert d.sizes[0][0] == 2
    d = _decide(_multi([0, 0], D=[8, 9], b_max=8))
    assert d.inst[0] == -1 and d.flags[0] == oracle.R_REJECT and d.hit[0] == 0


def test_packing_key_order():
    """Table 4's D-C-Q: most decoding first, then most cached, then fewest
    queued, then lowest id; all candidates feasible here."""
    big = dict(eta=1.0)
    # D dominates the hit
    assert _decide(_multi([8, 1], D=[1, 2], **big)).inst[0] == 1
    # equal D: hit decides
    assert _decide(_multi([5, 7], D=[2, 2], **big)).inst[0] == 1
    # equal D and hit: fewer queued
    assert _decide(_multi([5, 5], D=[2, 2], Q=[3, 1], **big)).inst[0] == 1
    # full tie: lowest id
    assert _decide(_multi([5, 5, 5], D=[2, 2, 2], Q=[1, 1, 1], **big)).inst[0] == 0


def test_fallback_lmetric_product():
    """Fallback = min (P_i + n_i)(A_i + 1) over C (LMetric, Sec. 8.1);
    L = 128 tokens.  Products: (100+128)*1 = 228, (0+64)*4 = 256,
    (200+0)*1 = 200 -> instance 2."""
    d = _decide(_multi([0, 4, 8], D=[0, 2, 0], Q=[0, 1, 0], P=[100, 0, 200], eta=1.0,
                       tpot_slo=1e-9))
    assert d.flags[0] & oracle.R_FALLBACK and d.inst[0] == 2
    # tie on the product -> lowest id: (64+64)*1 = 128 and (0+64)*2 = 128
    d = _decide(_multi([4, 4], D=[0, 1], P=[64, 0], eta=1.0, tpot_slo=1e-9))
    assert d.inst[0] == 0


def test_walk_stops_at_first_miss():
    """Longest cached prefix: a set holding every block but the second gives
    hit 1, not 7 (non-prefix-closed set)."""
    ch = chain_hashes(8)
    w = make_window([[ch[0]] + ch[2:]], [ch], [0], [0], [0], [0], SIMPLE_ALPHA, (64,),
                    ((0.01, 0, 0),), (1.0,), cap=8, tpot_slo=10.0)
    assert _decide(w).hit[0] == 1
    o = oracle.Oracle.from_window(w)
    assert o.window_hits(w)[0, 0] == 1


# -- brute force at the token level -----------------------------------------

def _block_hashes(tokens, bs=16):
    h = b"\0" * 8
    out = []
    for j in range(len(tokens) // bs):
        m = hashlib.blake2b(h + np.asarray(tokens[j * bs:(j + 1) * bs], np.int64).tobytes(),
                            digest_size=8)
        h = m.digest()
        v = int.from_bytes(h, "little") or 1
        out.append(v)
    return out


def test_hits_match_token_level_lcp():
    """hit = floor(max over cached sequences of LCP(request tokens, seq) / 16),
    with near-miss blocks that share 15 of 16 tokens."""
    rng = np.random.default_rng(7)
    bs = 16
    for trial in range(6):
        base = [list(rng.integers(0, 50, size=bs * rng.integers(2, 10))) for _ in range(5)]
        cached = []   # per instance: list of token sequences
        for i in range(4):
            seqs = []
            for _ in range(rng.integers(1, 4)):
                b = base[rng.integers(0, len(base))]
                cut = int(rng.integers(0, len(b) // bs + 1)) * bs
                s = list(b[:cut])
                if cut and rng.random() < 0.5:
                    # near miss: change one token of the last block
                    s[cut - 1 - int(rng.integers(0, bs))] += 1000
                seqs.append(s)
            cached.append(seqs)
        reqs = []
        for _ in range(8):
            b = base[rng.integers(0, len(base))]
            k = int(rng.integers(1, len(b) // bs + 1)) * bs
            r = list(b[:k]) + list(rng.integers(100, 200, size=bs * int(rng.integers(0, 3))))
            reqs.append(r)
        sets = [sorted({h for s in seqs for h in _block_hashes(s)}) for seqs in cached]
        chains = [_block_hashes(r) for r in reqs]
        w = make_window(sets, chains, [0] * 4, [0] * 4, [0] * 4, [0] * 4, SIMPLE_ALPHA, (64,),
                        ((0.01, 0, 0),), (1.0,), cap=max(len(s) for s in sets) + 1)
        o = oracle.Oracle.from_window(w)
        got = o.window_hits(w)
        for r, toks in enumerate(reqs):
            for i, seqs in enumerate(cached):
                best = 0
                for s in seqs:
                    lcp = 0
                    while lcp < min(len(s), len(toks)) and s[lcp] == toks[lcp]:
                        lcp += 1
                    best = max(best, lcp // bs)
                assert got[r, i] == best, (trial, r, i)


# -- generator construction (closed form of the owner hit) -------------------

@pytest.mark.parametrize("name,n_req", [("c1", 1024), ("c2", 2048), ("c3", 256)])
def test_hits_match_generator_construction(name, n_req):
    """Owner hit = min(P_s + 8k, cached prefix of the session), widened by a
    shared system prompt held on the instance; every other instance hits only
    the system prompt (or nothing)."""
    gen = {"c3": dict(n_inst=64, n_sess=512)}.get(name, {})
    w = synth.generate(name, n_req=n_req, **gen)
    o = oracle.Oracle.from_window(w)
    hits = o.window_hits(w)
    m = w.meta
    for r in range(w.n_req):
        s = m["req_sess"][r]
        pre = w.pre_len[r]
        sp = m["sess_sp"][s]
        for i in range(w.n_inst):
            have = m["inst_sp_have"][i] if sp else 0
            own = m["sess_cached_eff"][s] if i == m["sess_owner"][s] else 0
            assert hits[r, i] == min(pre, max(own, have)), (r, i)


def test_hit_invariants_c2():
    """hit <= chain length; monotone along a session's steps."""
    w = synth.generate("c2", n_req=4096)
    o = oracle.Oracle.from_window(w)
    hits = o.window_hits(w)
    ell = (w.pre_len + w.tail_len).astype(np.int64)
    assert (hits <= ell[:, None]).all()
    sess, step = w.meta["req_sess"], w.meta["req_step"]
    order = np.lexsort((step, sess))
    hs, ss = hits[order], sess[order]
    same = ss[1:] == ss[:-1]
    assert (hs[1:][same] >= hs[:-1][same]).all()


# -- invariants of Algorithm 1 on generated windows --------------------------

def _check_decisions(w, d, hits):
    D, Q, P = w.D.astype(np.int64), w.Q.astype(np.int64), w.P
    nA, nC, nT = d.sizes[:, 0], d.sizes[:, 1], d.sizes[:, 2]
    assert (nT <= nC).all() and (nC <= nA).all()
    rej = d.inst < 0
    assert ((nA == 0) == rej).all()
    assert (d.flags[rej] == oracle.R_REJECT).all() and (d.hit[rej] == 0).all()
    fb = (d.flags & oracle.R_FALLBACK) != 0
    assert ((nT == 0) & ~rej == fb).all()
    ok = ~rej
    assert (d.hit[ok] == hits[ok, d.inst[ok]]).all()


def test_decision_invariants_and_monotonicity():
    w = synth.generate("c2", n_req=2048)
    o = oracle.Oracle.from_window(w)
    hits = o.window_hits(w).astype(np.int64)
    prev = None
    for eta in (0.0, 0.25, 0.5, 1.0):
        d = o.window_score(w, eta=eta)
        _check_decisions(w, d, hits)
        if prev is not None:
            assert (d.sizes[:, 1] >= prev.sizes[:, 1]).all()
        prev = d
    prev = None
    for tau in (0.01, 0.03, 0.05, 0.2):
        d = o.window_score(w, tpot_slo=tau)
        _check_decisions(w, d, hits)
        if prev is not None:
            assert (d.sizes[:, 2] >= prev.sizes[:, 2]).all()
            assert (d.sizes[:, 1] == prev.sizes[:, 1]).all()
        prev = d
    # the packing choice is in T and beats every other member of T on the
    # D-C-Q key; a fallback choice is in C
    d = o.window_score(w)
    m = oracle.model_of(w)
    eta = float(np.float32(w.policy["eta"]))
    tau = float(np.float32(w.policy["tpot_slo"]))
    for r in range(0, w.n_req, 17):
        ex = o.explain(m, w.chain(r))
        i = d.inst[r]
        assert ex["choice"] == i
        if i < 0:
            assert ex["elig"].sum() == 0
            continue
        T = np.nonzero(ex["inT"])[0]
        C = np.nonzero(ex["inC"])[0]
        assert set(T) <= set(C) <= set(np.nonzero(ex["elig"])[0])
        if not d.flags[r] & oracle.R_FALLBACK:
            assert i in T
            for j in T:
                assert (-int(w.D[i]), -int(ex["hit"][i]), int(w.Q[i]), i) <= \
                       (-int(w.D[j]), -int(ex["hit"][j]), int(w.Q[j]), j)
        else:
            assert len(T) == 0 and i in C
        # C is exactly {rho <= eta}; T exactly {TPOT < tau} within C
        el = ex["elig"] == 1
        assert (ex["inC"][el] == (ex["rho"][el] <= eta)).all()
        assert (ex["inT"][el] == (ex["inC"][el] & (ex["tpot"][el] < tau))).all()


def test_relabelling_equivariance():
    """Permuting instance ids permutes decisions, except where the lowest-id
    tie-break is what decided (then the keys of both choices are equal)."""
    w = synth.generate("c1")
    o = oracle.Oracle.from_window(w)
    d = o.window_score(w)
    perm = np.random.default_rng(3).permutation(w.n_inst)   # new id of old i = perm[i]
    inv = np.argsort(perm)
    w2 = synth.generate("c1")
    rows = [w.blk[w.blk_off[i]:w.blk_off[i + 1]] for i in inv]
    w2.blk_off = np.concatenate([[0], np.cumsum([len(x) for x in rows])]).astype(np.int64)
    w2.blk = np.concatenate(rows).astype(np.uint64)
    for k in ("D", "Q", "P", "S"):
        setattr(w2, k, getattr(w, k)[inv].copy())
    o2 = oracle.Oracle.from_window(w2)
    d2 = o2.window_score(w2)
    hits = o.window_hits(w)
    for r in range(w.n_req):
        a, b = d.inst[r], d2.inst[r]
        if a < 0:
            assert b < 0
            continue
        if perm[a] == b:
            continue
        b_old = inv[b]
        if d.flags[r] & oracle.R_FALLBACK:
            L = int(w.pre_len[r] + w.tail_len[r]) * 16
            pa = (int(w.P[a]) + L - 16 * int(hits[r, a])) * (int(w.D[a]) + int(w.Q[a]) + 1)
            pb = (int(w.P[b_old]) + L - 16 * int(hits[r, b_old])) * (int(w.D[b_old]) + int(w.Q[b_old]) + 1)
            assert pa == pb
        else:
            assert (w.D[a], hits[r, a], w.Q[a]) == (w.D[b_old], hits[r, b_old], w.Q[b_old])


# -- commit (sequential state update) ----------------------------------------

def test_commit_hand_trace():
    ch = chain_hashes(6)
    other = chain_hashes(3, base=50_000)
    # instance 0 holds the first 2 blocks; instance 1 holds nothing; cap 5
    w = make_window([ch[:2], []], [ch, ch, other], [1, 0], [0, 2], [10, 20], [100, 200],
                    SIMPLE_ALPHA, (64,), ((0.01, 0, 0),), (1.0,), cap=5)
    o = oracle.Oracle.from_window(w)
    dropped = o.commit(w.pool, w.pre_off, w.pre_len, w.tail_off, w.tail_len, [0, -1, 0])
    st = o.state()
    # entry 0: L = 96, hit 2 -> n = 64 tokens; blocks 3..5 enter (set size 5 =
    # cap) and block 6 is refused; entry 1: skipped; entry 2: L = 48, hit 0 ->
    # n = 48, all 3 blocks refused
    assert list(st["Q"]) == [2, 2]
    assert list(st["P"]) == [10 + 64 + 48, 20]
    assert list(st["S"]) == [100 + 96 + 48, 200]
    assert list(st["set_size"]) == [5, 0] and dropped == 1 + 3
    h = o.window_hits(w)
    assert list(h[:, 0]) == [5, 5, 0]


# -- policy variants: selector orders (Table 4) and admission layers (Table 3)

def _sel_window(**pol):
    """Four instances all in T (no prefill cost, so no KVC effect; tau large).
    hits 2, 1, 3, 8; D 5, 5, 5, 4; Q 2, 1, 1, 0; S 1000, 5000, 3000, 2000."""
    ch = chain_hashes(8)
    hits = [2, 1, 3, 8]
    pol.setdefault("tpot_slo", 10.0)
    pol.setdefault("b_max", 10_000)
    pol.setdefault("kv_cap_tokens", 10**9)
    return make_window([ch[:h] for h in hits], [ch], [5, 5, 5, 4], [2, 1, 1, 0], [0, 0, 0, 0],
                       [1000, 5000, 3000, 2000], [0.0] * 6, (10_000,), ((0.01, 0.0, 1e-6),),
                       (1.0,), cap=8, lout=1e9, **pol)


def test_selector_orders():
    """D: most decoding then lowest id -> 0.  D-Q: then fewest queued -> 1.
    D-C and D-Q-C and D-C-Q: then most cached -> 2 (D-Q-C: Q ties 1, 2 ->
    hit 3 wins).  LMetric (P + n)(A + 1): 96*8, 112*7, 80*7, 0*5 -> 3.
    H-C-Q: smallest headroom tau - TPOT = largest TPOT = largest S -> 1."""
    want = {oracle.SEL_D: 0, oracle.SEL_DQ: 1, oracle.SEL_DC: 2, oracle.SEL_DQC: 2,
            oracle.SEL_DCQ: 2, oracle.SEL_LMETRIC: 3, oracle.SEL_HCQ: 1}
    for sel, inst in want.items():
        d = _decide(_sel_window(flags=oracle.selector_flags(sel)))
        assert d.inst[0] == inst, sel
        assert d.sizes[0][2] == 4 and not d.flags[0] & oracle.R_FALLBACK


def test_selector_dq_vs_dqc_order_of_ties():
    """D-Q-C compares queued before cached, D-C-Q cached before queued:
    instances (D, Q, hit) = (5, 2, 7) and (5, 1, 3) split them."""
    ch = chain_hashes(8)
    w = make_window([ch[:7], ch[:3]], [ch], [5, 5], [2, 1], [0, 0], [0, 0], [0.0] * 6,
                    (10_000,), ((0.01, 0.0, 0.0),), (1.0,), cap=8, tpot_slo=10.0, b_max=100,
                    kv_cap_tokens=10**9)
    assert _decide(w, flags=oracle.selector_flags(oracle.SEL_DCQ)).inst[0] == 0
    assert _decide(w, flags=oracle.selector_flags(oracle.SEL_DQC)).inst[0] == 1


def test_random_selector_uses_splitmix64_stream():
    """k = floor(z_hi * |T| / 2^32), z = the (r + 1)-th SplitMix64 output of
    the stream seeded with rand_seed (published definition; the generator's
    splitmix64 is checked against the reference vector in test_synth)."""
    gamma = 0x9E3779B97F4A7C15
    for seed in (0, 1, 12345, 2**63 + 7):
        w = _sel_window(flags=oracle.selector_flags(oracle.SEL_RANDOM), rand_seed=seed)
        z = synth.splitmix64(seed)                       # r = 0: state seed + gamma
        k = ((z >> 32) * 4) >> 32
        d = _decide(w)
        assert d.inst[0] == [0, 1, 2, 3][k], seed
    # request index r uses the (r + 1)-th output
    ch = chain_hashes(8)
    w = _sel_window(flags=oracle.selector_flags(oracle.SEL_RANDOM), rand_seed=99)
    w2 = make_window([ch[:h] for h in [2, 1, 3, 8]], [ch, ch, ch], [5, 5, 5, 4], [2, 1, 1, 0],
                     [0] * 4, [1000, 5000, 3000, 2000], [0.0] * 6, (10_000,),
                     ((0.01, 0.0, 1e-6),), (1.0,), cap=8, lout=1e9, tpot_slo=10.0, b_max=10_000,
                     kv_cap_tokens=10**9, flags=oracle.selector_flags(oracle.SEL_RANDOM),
                     rand_seed=99)
    d = _decide(w2)
    for r in range(3):
        z = synth.splitmix64((99 + r * gamma) & 0xFFFFFFFFFFFFFFFF)
        assert d.inst[r] == ((z >> 32) * 4) >> 32


def _layer_window(tau, **pol):
    """T_pf = N, so W = n and rho = n / 128 (L = 128): hits 8, 0, 6 give
    rho 0, 1, 0.25; eta = 0.5 -> C = {0, 2}.  Decode 0.01 + 1e-6 (S + 128)
    with S = 20000, 1000, 2000 -> TPOT 0.0301, 0.0111, 0.0121 (interference
    is negligible: L_out = 1e9).  D = 1, 9, 3; P = 0."""
    ch = chain_hashes(8)
    return make_window([ch, [], ch[:6]], [ch], [1, 9, 3], [0, 0, 0], [0, 0, 0],
                       [20000, 1000, 2000], [0, 1.0, 0, 0, 0, 0], (10_000,),
                       ((0.01, 0.0, 1e-6),), (1.0,), cap=8, lout=1e9, eta=0.5, tpot_slo=tau,
                       b_max=10_000, kv_cap_tokens=10**9, **pol)


def test_admission_layers_table3():
    """G = capacity only, C = cache only, T = TPOT only (DCQ fallback over A),
    CT = cache + TPOT (DCQ fallback over C), F = full (LMetric fallback)."""
    G = oracle.F_NO_KVC_FILTER | oracle.F_NO_TPOT_FILTER
    C = oracle.F_NO_TPOT_FILTER
    T = oracle.F_NO_KVC_FILTER | oracle.F_FALLBACK_DCQ
    CT = oracle.F_FALLBACK_DCQ
    F = 0
    # tau = 0.02: T passes instances 1 and 2
    want = {G: (1, False), C: (2, False), T: (1, False), CT: (2, False), F: (2, False)}
    for fl, (inst, fb) in want.items():
        d = _decide(_layer_window(0.02, flags=fl))
        assert d.inst[0] == inst and bool(d.flags[0] & oracle.R_FALLBACK) == fb, fl
    # tau = 0.001: nobody passes TPOT; fallbacks: F -> LMetric over C
    # (n (A + 1) = 0 * 2 for instance 0), CT -> D-C-Q over C (instance 2),
    # T -> D-C-Q over A (instance 1)
    want = {T: 1, CT: 2, F: 0}
    for fl, inst in want.items():
        d = _decide(_layer_window(0.001, flags=fl))
        assert d.inst[0] == inst and d.flags[0] & oracle.R_FALLBACK, fl


def test_headroom_near_tie_is_flagged():
    """H-C-Q: two members of T whose headrooms agree to 1e-5 tau are a
    near-boundary decision (their order is decided by rounding)."""
    ch = chain_hashes(8)
    w = make_window([ch[:2], ch[:3]], [ch], [5, 5], [0, 0], [0, 0], [1000, 1000], [0.0] * 6,
                    (10_000,), ((0.01, 0.0, 1e-6),), (1.0,), cap=8, tpot_slo=10.0, b_max=100,
                    kv_cap_tokens=10**9, lout=1e9, flags=oracle.selector_flags(oracle.SEL_HCQ))
    d = _decide(w)
    assert d.inst[0] == 1 and d.nb[0] & oracle.NB_HEADROOM


# -- near-boundary rule: which comparisons rounding may decide ---------------
# The parity tests exclude a decision from the exact check only where the
# oracle marks it; these pins fix each mark's window (1e-5 relative: inside
# at 0.5e-5, outside at 2e-5) and where it applies.

NB_ALL_DEC = oracle.NB_DECISION


def _nb_tpot_window(S, tau, D=None, hits=None, eta=0.5):
    """Instances with nothing queued and A = 0 unless D is given, a 128-token
    request, decode time t_iter = 0.5 + 1e-6 (S + 128) (no interference on an
    idle instance), so TPOT is set by S; alpha of the simple model."""
    n = len(S)
    ch = chain_hashes(8)
    hits = hits if hits is not None else [0] * n
    return make_window([ch[:h] for h in hits], [ch], D if D is not None else [0] * n, [0] * n,
                       [0] * n, S, SIMPLE_ALPHA, (10_000,), ((0.5, 0.0, 1e-6),), (1.0,), cap=8,
                       tpot_slo=tau, eta=eta, b_max=10_000, kv_cap_tokens=10**9, lout=556.0)


def test_nb_tpot_window():
    """One idle instance, TPOT = 0.500128: tau 0.5e-5 above or below it marks
    the decision (the choice itself, or an empty T whose fallback it would
    replace), 2e-5 away marks nothing."""
    tp = 0.5 + 1e-6 * 128
    for rel, marked in ((0.5e-5, True), (-0.5e-5, True), (2e-5, False), (-2e-5, False)):
        d = _decide(_nb_tpot_window([0], tp * (1 + rel)))
        assert bool(d.nb[0] & oracle.NB_TPOT) == marked, rel
        assert bool(d.nb[0] & oracle.NB_SIZES) == marked, rel
        assert d.nb[0] >> oracle.NB_UNSURE_SHIFT == (1 if marked else 0), rel
        assert d.nb[0] & (NB_ALL_DEC & ~oracle.NB_TPOT) == 0, rel
        assert bool(d.flags[0] & oracle.R_FALLBACK) == (rel < 0), rel


def test_nb_tpot_only_where_it_can_change_the_decision():
    """tau = 1.  Instance 0 (TPOT 0.500128) is the choice; a second instance
    with TPOT within 1e-5 of tau (S = 499,872: TPOT = 1.0) that comes after it
    in key order moves only |T| (NB_SIZES, one unsure candidate); placed
    first in key order it could be the choice (NB_TPOT); outside C (eta = 0,
    hit 0 against a full hit) it is not counted at all."""
    d = _decide(_nb_tpot_window([0, 499_872], 1.0))
    assert d.inst[0] == 0 and d.nb[0] & NB_ALL_DEC == 0
    assert d.nb[0] & oracle.NB_SIZES and d.nb[0] >> oracle.NB_UNSURE_SHIFT == 1
    d = _decide(_nb_tpot_window([0, 499_872 - 2], 1.0))     # inside T, not the choice
    assert d.inst[0] == 0 and d.nb[0] & NB_ALL_DEC == 0 and d.nb[0] & oracle.NB_SIZES
    d = _decide(_nb_tpot_window([499_872, 0], 1.0))         # first in key order
    assert d.inst[0] == 1 and d.nb[0] & oracle.NB_TPOT
    d = _decide(_nb_tpot_window([0, 499_872], 1.0, hits=[8, 0], eta=0.0))   # not in C
    assert d.inst[0] == 0 and list(d.sizes[0]) == [2, 1, 1] and d.nb[0] == 0


def _nb_ttft_window(floor, Q=1, flags=0):
    """One instance, alpha = (0.5, 1e-3, 0, ...), a 128-token request with
    nothing cached: T_pf(128, 0) = 0.628, Z = 0.128, TTFT = 0.628 + 0.5 Q.
    The budget is the floor (above 0.628) unless the floor is lower."""
    ch = chain_hashes(8)
    return make_window([[]], [ch], [0], [Q], [0], [0], [0.5, 1e-3, 0, 0, 0, 0], (10_000,),
                       ((0.01, 0.0, 0.0),), (1.0,), cap=8, tpot_slo=10.0, ttft_floor=floor,
                       b_max=100, kv_cap_tokens=10**9, flags=flags)


def test_nb_ttft_admission_window():
    """TTFT admission on, TTFT = 1.128: a budget within 0.5e-5 of it marks
    the decision (NB_TTFT), 2e-5 away marks nothing."""
    tt = 0.628 + 0.5
    for rel, marked in ((0.5e-5, True), (-0.5e-5, True), (2e-5, False), (-2e-5, False)):
        d = _decide(_nb_ttft_window(tt * (1 + rel), flags=oracle.F_TTFT_ADMIT))
        assert bool(d.nb[0] & oracle.NB_TTFT) == marked, rel
        assert d.nb[0] & (NB_ALL_DEC & ~oracle.NB_TTFT) == 0, rel
        assert bool(d.flags[0] & oracle.R_FALLBACK) == (rel < 0), rel
        # without admission TTFT decides nothing
        d = _decide(_nb_ttft_window(tt * (1 + rel)))
        assert d.nb[0] & NB_ALL_DEC == 0 and not d.flags[0] & oracle.R_FALLBACK, rel


def test_nb_ttft_miss_flag_window():
    """The chosen instance's TTFT_MISS flag (TTFT above the budget): within
    0.5e-5 of the budget it is marked (NB_MISSFLAG), 2e-5 away it is not,
    and in neither case is the decision marked."""
    tt = 0.628 + 0.5
    for rel, marked in ((0.5e-5, True), (-0.5e-5, True), (2e-5, False), (-2e-5, False)):
        d = _decide(_nb_ttft_window(tt * (1 + rel)))
        assert bool(d.nb[0] & oracle.NB_MISSFLAG) == marked, rel
        assert d.nb[0] & NB_ALL_DEC == 0, rel
        assert bool(d.flags[0] & oracle.R_TTFT_MISS) == (rel < 0), rel


def test_nb_ttft_equal_to_budget_by_construction():
    """Nothing cached, nothing queued and the budget T_pf(L, 0) above the
    floor: TTFT is the budget itself, so the comparison is exact in any
    precision and marks nothing (no TTFT_MISS, admitted under admission)."""
    for flags in (0, oracle.F_TTFT_ADMIT):
        d = _decide(_nb_ttft_window(0.1, Q=0, flags=flags))
        assert d.ttft[0] == pytest.approx(0.628, rel=1e-12)
        assert d.nb[0] == 0 and d.flags[0] == 0, flags


def test_nb_rho_window():
    """T_pf = N makes rho = 1/2 exactly for hits 8 and 4 of 8 blocks: eta
    within 0.5e-5 of it marks the decision, 3e-5 away does not."""
    alpha = [0, 1.0, 0, 0, 0, 0]
    for off, marked in ((0.5e-5, True), (-0.5e-5, True), (3e-5, False), (-3e-5, False)):
        d = _decide(_multi([8, 4], alpha=alpha, eta=0.5 + off, D=[0, 5]))
        assert bool(d.nb[0] & oracle.NB_RHO) == marked, off
        assert d.inst[0] == (1 if off > 0 else 0), off


def test_nb_rho_one_by_construction():
    """A fully cached candidate makes W_min = 0 exactly, and a candidate with
    nothing cached has W = Z: its rho is exactly 1 in any precision, so eta
    = 1 keeps it unmarked (and in C); eta = 1 + 0.5e-5 still marks nothing,
    while a partly cached minimiser leaves the zero-hit rho = 1 - W_min / Z
    to rounding only near eta."""
    for eta in (1.0, 1.0 + 0.5e-5):
        d = _decide(_multi([8, 0, 0], D=[0, 5, 0], eta=eta))
        assert d.nb[0] == 0 and list(d.sizes[0][:2]) == [3, 3] and d.inst[0] == 1, eta
    d = _decide(_multi([8, 0], alpha=[0, 1.0, 0, 0, 0, 0], eta=1.0 + 0.5e-5, D=[0, 5]))
    assert d.nb[0] == 0 and d.inst[0] == 1
    d = _decide(_multi([4, 0], alpha=[0, 1.0, 0, 0, 0, 0], eta=0.5 + 0.5e-5, D=[0, 5]))
    assert d.nb[0] & oracle.NB_RHO


def test_nb_zero_benefit_window():
    """Z = a1 L with T_pf(L, 0) = 0.02 + a1 L: Z within 1e-5 of T_pf(L, 0)
    marks the decision, 3e-5 does not."""
    for z_rel, marked in ((0.5e-5, True), (3e-5, False)):
        a1 = 0.02 * z_rel / (1 - z_rel) / 128
        d = _decide(_multi([0, 3, 5, 8], alpha=[0.02, a1, 0, 0, 0, 0], eta=0.0))
        assert bool(d.nb[0] & oracle.NB_Z) == marked, z_rel


def _follow_window():
    """Two idle instances and one at its batch limit, no cache, two requests
    with the same 8-block chain; tau within 1e-5 above instance 0's TPOT, so
    the first decision (instance 0) is near its boundary; instance 1 is
    far above tau."""
    ch = chain_hashes(8)
    tp0 = 0.5 + 1e-6 * 128
    return make_window([[], [], []], [ch, ch], [0, 0, 10], [0, 0, 0], [0, 0, 0], [0, 50_000, 0],
                       SIMPLE_ALPHA, (10_000,), ((0.5, 0.0, 1e-6),), (1.0,), cap=64,
                       tpot_slo=tp0 * (1 + 0.5e-5), eta=0.0, b_max=10, kv_cap_tokens=10**9)


def test_schedule_follows_only_near_boundary_decisions():
    """Per arrival with another implementation's placements: at the first
    request (near the TPOT boundary) the oracle commits the followed
    instance 1, so the second request finds its blocks there (hit 8, the
    only member of C at eta = 0, TPOT above tau: fallback); at the second
    request (not near a boundary) a different followed placement is
    ignored.  Without placements to follow both go to instance 0; a
    followed instance outside A is refused."""
    w = _follow_window()
    o = oracle.Oracle.from_window(w)
    d, _ = o.window_schedule(w)
    assert list(d.inst) == [0, 0] and list(d.hit) == [0, 8]
    assert d.nb[0] & oracle.NB_TPOT and d.nb[1] & NB_ALL_DEC == 0
    o = oracle.Oracle.from_window(w)
    d, _ = o.window_schedule(w, follow=[1, 0])
    assert list(d.inst) == [0, 1] and list(d.hit) == [0, 8]
    assert d.flags[1] & oracle.R_FALLBACK and d.nb[1] & NB_ALL_DEC == 0
    assert list(o.state()["Q"]) == [0, 2, 0]
    o = oracle.Oracle.from_window(w)
    with pytest.raises(ValueError):
        o.window_schedule(w, follow=[2, 0])


# -- feedback path: EMA calibration (Sec. 5.3), median output, transitions ----

def _fb_model(gamma=(1.0, 1.0)):
    return oracle.make_model([0.02, 1e-4, 0, 0, 0, 0], (8, 64), ((0.01, 1e-3, 1e-6), (0.02, 0.0, 0.0)),
                             gamma, 0.5, 0.05, 2.0, 556.0, 16, 64, 10**6)


def test_ema_update_rule():
    """Factor f of the sample's segment: f <- clip(0.98 f + 0.02 clip(ratio,
    0.5, 2), 1, 2), ratio = measured / (b0 + b1 B + b2 S) of the base model.
    Segment 0 (B <= 8): prediction 0.01 + 0.001*4 + 1e-6*6000 = 0.02."""
    m = _fb_model()
    oracle.feedback_decode(m, [4], [6000], [0.03])          # ratio 1.5
    assert m.gamma[0] == pytest.approx(0.98 + 0.03, rel=1e-12) and m.gamma[1] == 1.0
    oracle.feedback_decode(m, [4], [6000], [0.2])           # ratio 10 -> clipped to 2
    assert m.gamma[0] == pytest.approx(0.98 * 1.01 + 0.04, rel=1e-12)
    m = _fb_model()
    oracle.feedback_decode(m, [4], [6000], [0.001])         # ratio 0.05 -> 0.5; factor floor 1
    assert m.gamma[0] == 1.0
    m = _fb_model((2.0, 1.0))
    oracle.feedback_decode(m, [4], [6000], [0.04])          # ratio 2 keeps 2 (ceiling)
    assert m.gamma[0] == 2.0
    m = _fb_model()
    oracle.feedback_decode(m, [20], [0], [0.03])            # B = 20 -> segment 1, pred 0.02
    assert m.gamma[1] == pytest.approx(1.01, rel=1e-12) and m.gamma[0] == 1.0
    m = _fb_model()
    oracle.feedback_decode(m, [4] * 2000, [6000] * 2000, [0.04] * 2000)
    assert 1.99 < m.gamma[0] <= 2.0                        # converges to the clipped ratio


def test_median_output_tracker():
    w = synth.generate("c1", n_req=4)
    o = oracle.Oracle.from_window(w)
    m = oracle.model_of(w)
    o.feedback_output(m, [5, 1, 3])
    assert m.lout == 3.0                                    # sorted 1 3 5
    o.feedback_output(m, [4])
    assert m.lout == 3.0                                    # 1 3 4 5 -> lower median 3
    o2 = oracle.Oracle.from_window(w)
    m2 = oracle.model_of(w)
    o2.feedback_output(m2, list(range(1, 1101)))            # keeps the last 1024: 77..1100
    assert m2.lout == 77 + 511


def test_event_transitions():
    w = synth.generate("c1", n_req=4)
    o = oracle.Oracle.from_window(w)
    st0 = o.state()
    i = int(np.argmax(st0["Q"]))
    assert o.apply_events([i, i, i], [1, 2, 3], [100, 5000, 3000]) == 0
    st = o.state()
    assert st["Q"][i] == st0["Q"][i] - 1 and st["D"][i] == st0["D"][i]
    assert st["P"][i] == st0["P"][i] - 100 and st["S"][i] == st0["S"][i] + 2000
    # all or nothing: the second event would drive D below zero
    j = int(np.argmin(st["D"]))
    before = o.state()
    assert o.apply_events([i, j] + [j] * (int(st["D"][j]) + 1), [2, 3] + [3] * (int(st["D"][j]) + 1),
                          [1] * (int(st["D"][j]) + 3)) == -5
    after = o.state()
    for k in ("D", "Q", "P", "S"):
        assert (before[k] == after[k]).all()
    assert o.apply_events([0], [7], [0]) == -1


# -- Algorithm 1 per arrival (each placement changes the state the next
#    request sees) and the replay of given placements

def _rr_window(n_inst=5, n_req=23, D=3, b_max=7):
    """Identical idle-queue instances (same D, nothing cached) and requests of
    four fresh blocks each (no block shared between requests)."""
    chains = [chain_hashes(4, base=10_000 * (k + 1)) for k in range(n_req)]
    return make_window([[] for _ in range(n_inst)], chains, [D] * n_inst, [0] * n_inst,
                       [0] * n_inst, [0] * n_inst, SIMPLE_ALPHA, (64,), ((0.01, 0.0, 0.0),),
                       (1.0,), cap=64, tpot_slo=10.0, b_max=b_max, kv_cap_tokens=10**9)


def test_sequential_round_robin_closed_form():
    """Equal D and no cache: each placement adds one to Q, so by D-C-Q the
    k-th request goes to instance k mod n.  With A = D + Q, an instance takes
    requests while A + 1 <= B_max, i.e. B_max - D = 4 of them; after n * 4
    placements A is empty and every later request is rejected.  |A| at
    request k of the last round, 15 + j, is n - j.  Against the snapshot all
    of them pick instance 0."""
    w = _rr_window()
    o = oracle.Oracle.from_window(w)
    d, dropped = o.window_schedule(w)
    want = [k % 5 for k in range(20)] + [-1, -1, -1]
    assert list(d.inst) == want
    assert list(d.hit) == [0] * 23 and dropped == 0
    nA = [5] * 15 + [5, 4, 3, 2, 1] + [0, 0, 0]
    assert list(d.sizes[:, 0]) == nA
    assert all(d.flags[20:] == oracle.R_REJECT)
    st = o.state()
    assert list(st["Q"]) == [4] * 5 and list(st["P"]) == [4 * 64] * 5
    assert list(st["S"]) == [4 * 64] * 5 and list(st["set_size"]) == [16] * 5
    snap = _decide(_rr_window())
    assert list(snap.inst) == [0] * 23


def _session_window():
    """Two instances with D = 2 and nothing cached; requests: session A's
    first 4 blocks, session B's first 4, A's first 6, B's first 5, and two
    blocks of a third session.  eta = 0: only minimum-penalty candidates
    pass the KVC-first stage."""
    a = chain_hashes(6, base=1_000)
    b = chain_hashes(5, base=2_000)
    c = chain_hashes(2, base=3_000)
    return make_window([[], []], [a[:4], b[:4], a, b, c], [2, 2], [0, 0], [0, 0], [0, 0],
                       SIMPLE_ALPHA, (64,), ((0.01, 0.0, 0.0),), (1.0,), cap=64, eta=0.0,
                       tpot_slo=10.0, b_max=100, kv_cap_tokens=10**9)


def test_sequential_session_follows_its_blocks():
    """Hand trace.  r0 (A, 4 blocks): tie -> instance 0; its blocks enter
    instance 0, Q0 = 1.  r1 (B, 4): hits 0 / 0, D-C-Q by Q -> instance 1.
    r2 (A, 6): hit 4 on instance 0, 0 on 1; eta = 0 keeps only instance 0.
    r3 (B, 5): hit 4 on instance 1 -> 1.  r4 (C, 2): Q0 = Q1 = 2 -> 0.
    r2's latencies on instance 0 (Q = 1, P = 64, S = 64): n = 32, c = 64
    tokens, T_pf = 0.02 + 0.032 + 0.002048 + 0.001024 + 0.00064 +
    0.000008192 = 0.055720192; TTFT = T_pf + 0.02 * 1 + 0.001 * 64;
    TPOT = 0.01 + T_pf / 556 (busy instance).  The snapshot sends every
    request to instance 0 with hit 0."""
    w = _session_window()
    o = oracle.Oracle.from_window(w)
    d, _ = o.window_schedule(w)
    assert list(d.inst) == [0, 1, 0, 1, 0]
    assert list(d.hit) == [0, 0, 4, 4, 0]
    tpf = 0.055720192
    assert d.ttft[2] == pytest.approx(tpf + 0.02 + 0.064, rel=1e-12)
    assert d.tpot[2] == pytest.approx(0.01 + tpf / 556.0, rel=1e-12)
    st = o.state()
    # P: instance 0 gets 64 + 32 + 32 new tokens, instance 1 gets 64 + 16
    assert list(st["Q"]) == [3, 2] and list(st["P"]) == [128, 80]
    assert list(st["S"]) == [64 + 96 + 32, 64 + 80] and list(st["set_size"]) == [8, 5]
    snap = _decide(_session_window())
    assert list(snap.inst) == [0] * 5 and list(snap.hit) == [0] * 5


def test_replay_hand_trace():
    """The snapshot's placements (all on instance 0) applied in arrival
    order, each measured in the state the earlier ones left:
      r0: hit 0, Q 0, P 0:    TTFT = T_pf(64, 0) = 0.088096
      r1: hit 0, Q 1, P 64:   TTFT = 0.088096 + 0.02 + 0.064
      r2: hit 4, Q 2, P 128:  TTFT = 0.055720192 + 0.04 + 0.128
      r3: hit 4, Q 3, P 160:  T_pf(16, 64) = 0.037928192, + 0.06 + 0.16
      r4: hit 0, Q 4, P 176:  T_pf(32, 0) = 0.053024, + 0.08 + 0.176
    TPOT = 0.01 plus the interference T_pf / 556 (D = 2: always busy)."""
    w = _session_window()
    o = oracle.Oracle.from_window(w)
    hit, ttft, tpot, dropped = o.window_replay(w, [0] * 5)
    assert list(hit) == [0, 0, 4, 4, 0] and dropped == 0
    tpf = [0.088096, 0.088096, 0.055720192, 0.037928192, 0.053024]
    want = [tpf[0], tpf[1] + 0.084, tpf[2] + 0.168, tpf[3] + 0.22, tpf[4] + 0.256]
    assert np.allclose(ttft, want, rtol=1e-12, atol=0)
    assert np.allclose(tpot, [0.01 + t / 556.0 for t in tpf], rtol=1e-12, atol=0)
    st = o.state()
    assert list(st["Q"]) == [5, 0] and list(st["P"]) == [176 + 32, 0]
    # skipped entries report zeros and change nothing
    o2 = oracle.Oracle.from_window(w)
    hit2, ttft2, _, _ = o2.window_replay(w, [-1, 1, -1, -1, -1])
    assert list(hit2) == [0] * 5 and ttft2[0] == 0.0 and ttft2[1] == pytest.approx(0.088096)
    assert list(o2.state()["Q"]) == [0, 1]


def test_sequential_placements_hold_at_arrival():
    """On a loaded generated window with a binding TPOT target: replaying the
    per-arrival placements reproduces their hits and latencies exactly, and
    every placement that is not a fallback meets the TPOT target in the state
    it arrived to.  The snapshot's placements, replayed the same way, break
    it (the herding that per-arrival scoring removes)."""
    w = synth.generate("c1", seed=3)
    pol = dict(tpot_slo=0.030, b_max=96)
    o = oracle.Oracle.from_window(w)
    d, dropped = o.window_schedule(w, **pol)
    o2 = oracle.Oracle.from_window(w)
    hit, ttft, tpot, dropped2 = o2.window_replay(w, d.inst, **pol)
    placed = d.inst >= 0
    assert placed.sum() > 0.9 * w.n_req
    assert np.array_equal(hit[placed], d.hit[placed]) and dropped2 == dropped
    assert np.array_equal(ttft[placed], d.ttft[placed])
    assert np.array_equal(tpot[placed], d.tpot[placed])
    tau = float(np.float32(0.030))
    ok = placed & ((d.flags & oracle.R_FALLBACK) == 0)
    assert (tpot[ok] < tau).all()
    for k in ("Q", "P", "S", "set_size"):
        assert np.array_equal(o.state()[k], o2.state()[k])
    snap = _decide(w, **pol)
    o3 = oracle.Oracle.from_window(w)
    _, _, tpot_s, _ = o3.window_replay(w, snap.inst, **pol)
    ok_s = (snap.inst >= 0) & ((snap.flags & oracle.R_FALLBACK) == 0)
    assert (tpot_s[ok_s] >= tau).sum() > 0
