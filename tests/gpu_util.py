"""Helpers shared by the GPU tests: marshal a generated window into the C ABI
and compare GPU decisions with the oracle's."""
import numpy as np

import oracle

NB_TOL = 1e-5  # relative tolerance on predicted latencies (fp32 vs fp64)


def gpu_model(win, **policy):
    import paper_2609_33224_amd as ps
    pol = dict(win.policy)
    pol.update(policy)
    return ps.make_model(win.alpha, win.seg_ub, win.beta, win.gamma, pol["eta"], pol["tpot_slo"],
                         pol["ttft_floor"], pol["lout"], pol["block_tokens"], pol["b_max"],
                         pol["kv_cap_tokens"], pol.get("flags", 0), pol.get("rand_seed", 0))


def load_window(scorer, win, **policy):
    scorer.load(win.n_inst, win.cap, win.blk_off, win.blk, win.D, win.Q, win.P, win.S,
                gpu_model(win, **policy))


def reqs_of(win):
    import paper_2609_33224_amd as ps
    return ps.pack_reqs(win.pre_off, win.pre_len, win.tail_off, win.tail_len)


# Edge-case windows: a smooth synthetic model (fp32 coefficients) and random
# load, with explicit per-instance block lists and request chains.
ALPHA = [0.02, 1e-4, 1.5e-9, 7.5e-10, 1e-7, 1e-14]
SEG_UB, BETA, GAMMA = (8, 64, 512), ((0.01, 1e-4, 1e-8),) * 3, (1.0, 1.1, 1.2)


def edge_window(sets, chains, pool=None, reqs=None, **kw):
    """Edge-case window from explicit block sets and chains, or (chains None)
    from an explicit pool and descriptors (pre_off, pre_len, tail_off,
    tail_len) that may share pool segments."""
    from tests.tinywin import make_window, make_window_pool
    n = len(sets)
    rng = np.random.default_rng(len(sets) * 7 + (len(chains) if chains is not None else len(reqs)))
    D = kw.pop("D", rng.integers(0, 64, n))
    Q = kw.pop("Q", rng.integers(0, 4, n))
    P = kw.pop("P", rng.integers(0, 8192, n) * (np.asarray(Q) > 0))
    S = kw.pop("S", rng.integers(0, 500_000, n))
    cap = kw.pop("cap", max(max((len(s) for s in sets), default=1), 1))
    kw.setdefault("tpot_slo", 0.05)
    kw.setdefault("b_max", 512)
    kw.setdefault("kv_cap_tokens", 4_194_304)
    if chains is None:
        w = make_window_pool(sets, pool, reqs, D, Q, P, S, ALPHA, SEG_UB, BETA, GAMMA, cap=cap, **kw)
    else:
        w = make_window(sets, chains, D, Q, P, S, ALPHA, SEG_UB, BETA, GAMMA, cap=cap, **kw)
    w.alpha = np.asarray(w.alpha, np.float32)
    w.beta = np.asarray(w.beta, np.float32)
    w.gamma = np.asarray(w.gamma, np.float32)
    return w


class DeviceWindow:
    """The window's pool and descriptors resident on the GPU."""

    def __init__(self, win):
        import paper_2609_33224_amd as ps
        import torch
        self.pool_len = len(win.pool)
        self.n_req = win.n_req
        self.d_pool = ps.to_device_u64(win.pool if len(win.pool) else np.zeros(1, np.uint64))
        self.d_reqs = ps.to_device_bytes(reqs_of(win) if win.n_req else
                                         np.zeros(1, ps.PS_REQ_DTYPE))
        self.d_out = torch.zeros(max(self.n_req, 1) * 20, dtype=torch.uint8, device="cuda")
        self.d_sizes = torch.zeros(max(self.n_req, 1) * 3, dtype=torch.int32, device="cuda")

    def score(self, scorer, with_sizes=True, fixed=False):
        """Results (and |A|, |C|, |T| unless with_sizes is False, which takes
        the kernel's path that does not count the sets); fixed: through the
        allocation-free entry point."""
        import paper_2609_33224_amd as ps
        import torch
        call = scorer.score_dev_fixed if fixed else scorer.score_dev
        call(self.d_pool, self.pool_len, self.d_reqs, self.n_req, self.d_out,
             self.d_sizes if with_sizes else None)
        torch.cuda.synchronize()
        res = ps.results_from_device(self.d_out)[:self.n_req]
        if not with_sizes:
            return res, None
        sizes = self.d_sizes.cpu().numpy().view(np.uint32).reshape(-1, 3)[:self.n_req]
        return res, sizes

    def schedule(self, scorer, with_sizes=True):
        """Algorithm 1 per arrival: (results, sizes or None, dropped)."""
        import paper_2609_33224_amd as ps
        import torch
        dropped = scorer.schedule_dev(self.d_pool, self.pool_len, self.d_reqs, self.n_req,
                                      self.d_out, self.d_sizes if with_sizes else None)
        torch.cuda.synchronize()
        res = ps.results_from_device(self.d_out)[:self.n_req]
        sizes = None
        if with_sizes:
            sizes = self.d_sizes.cpu().numpy().view(np.uint32).reshape(-1, 3)[:self.n_req]
        return res, sizes, dropped

    def replay(self, scorer, inst):
        """Given placements measured at arrival: (results, dropped)."""
        import paper_2609_33224_amd as ps
        import torch
        d_inst = torch.from_numpy(np.ascontiguousarray(inst, np.int32)).to("cuda")
        dropped = scorer.replay_dev(self.d_pool, self.pool_len, self.d_reqs, self.n_req, d_inst,
                                    self.d_out)
        torch.cuda.synchronize()
        return ps.results_from_device(self.d_out)[:self.n_req], dropped

    def hits(self, scorer, n_inst):
        import torch
        d_hits = torch.zeros(max(self.n_req, 1) * n_inst, dtype=torch.int32, device="cuda")
        scorer.hits_dev(self.d_pool, self.pool_len, self.d_reqs, self.n_req, d_hits)
        torch.cuda.synchronize()
        return d_hits.cpu().numpy().view(np.uint32).reshape(-1, n_inst)[:self.n_req]


def nb_cap(n_req):
    """Most near-boundary decisions a window of n_req requests may exclude
    from the exact check: 0.1% of its requests, at least 8.  (The oracle's
    synthetic windows have 0.00-0.06%.)"""
    return max(8, n_req // 1000)


def compare_decisions(res, sizes, od, idx=None, tol=NB_TOL, label="", max_nb=None):
    """GPU results vs oracle decisions (optionally the oracle holds only the
    requests `idx` of the GPU window).  Returns the near-boundary count,
    which must not exceed `max_nb` (default nb_cap(n)).

    * chosen instance, hit and flags: bit-exact except on requests whose
      decision the oracle marks near a boundary (NB_DECISION); the TTFT_MISS
      flag is skipped where the oracle marks that flag near its boundary;
    * |A|: exact on every request (integer capacity tests);
    * |C|: exact except where a recomputation-filter comparison is near its
      boundary (NB_SET_C);
    * |T|: within the number of candidates whose T membership the oracle
      marks as decided by rounding (nb >> 16), exact where that is 0;
    * TTFT / TPOT of the choice within `tol` relative (non-NB requests)."""
    if idx is not None:
        res = res[idx]
        sizes = sizes[idx] if sizes is not None else None
    n = len(od.inst)
    nb_dec = (od.nb & oracle.NB_DECISION) != 0
    nb_flag = (od.nb & oracle.NB_MISSFLAG) != 0
    n_dec = int(nb_dec.sum())
    cap = nb_cap(n) if max_nb is None else max_nb
    assert n_dec <= cap, f"{label}: {n_dec} near-boundary decisions excluded, more than {cap}"
    ok = ~nb_dec
    bad = np.nonzero(ok & ((res["instance"] != od.inst) | (res["hit_blocks"] != od.hit)))[0]
    assert len(bad) == 0, (
        f"{label}: {len(bad)} decisions differ, first r={bad[0]}: gpu "
        f"{res[bad[0]]} oracle inst={od.inst[bad[0]]} hit={od.hit[bad[0]]} "
        f"flags={od.flags[bad[0]]} sizes={od.sizes[bad[0]]} nb={od.nb[bad[0]]:#x}"
        + (f" gpu sizes={sizes[bad[0]]}" if sizes is not None else ""))
    fl_mask = np.where(nb_flag, ~np.uint32(oracle.R_TTFT_MISS), np.uint32(0xFFFFFFFF))
    fbad = np.nonzero(ok & ((res["flags"] & fl_mask) != (od.flags & fl_mask)))[0]
    assert len(fbad) == 0, f"{label}: flags differ at r={fbad[:5]}"
    if sizes is not None:
        sizes = np.asarray(sizes, np.int64)
        want = od.sizes.astype(np.int64)
        abad = np.nonzero(sizes[:, 0] != want[:, 0])[0]
        assert len(abad) == 0, f"{label}: |A| differs at r={abad[:5]}: {sizes[abad[0]]} vs {want[abad[0]]}"
        c_ok = (od.nb & oracle.NB_SET_C) == 0
        cbad = np.nonzero(c_ok & (sizes[:, 1] != want[:, 1]))[0]
        assert len(cbad) == 0, f"{label}: |C| differs at r={cbad[:5]}: {sizes[cbad[0]]} vs {want[cbad[0]]}"
        unsure = (od.nb >> oracle.NB_UNSURE_SHIFT).astype(np.int64)
        tbad = np.nonzero(c_ok & (np.abs(sizes[:, 2] - want[:, 2]) > unsure))[0]
        assert len(tbad) == 0, (f"{label}: |T| differs at r={tbad[:5]}: {sizes[tbad[0]]} vs "
                                f"{want[tbad[0]]} ({unsure[tbad[0]]} unsure)")
    chosen = ok & (od.inst >= 0)
    for name, ref in (("ttft", od.ttft), ("tpot", od.tpot)):
        g = res[name][chosen].astype(np.float64)
        r = ref[chosen]
        rel = np.abs(g - r) / np.maximum(np.abs(r), 1e-30)
        assert (rel <= tol).all(), f"{label}: {name} rel err {rel.max():.3g} > {tol}"
    return n_dec


def compare_sequential(res, sizes, od, tol=NB_TOL, label="", max_nb=None):
    """Per-arrival results against the oracle's schedule run with
    follow=res["instance"] (so the oracle committed the GPU's placement
    wherever its own decision was near a boundary and they differ, and both
    went on from the same state).  Every request is compared as by
    compare_decisions; returns the number of near-boundary requests."""
    return compare_decisions(res, sizes, od, tol=tol, label=label, max_nb=max_nb)
