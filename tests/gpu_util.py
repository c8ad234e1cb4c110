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

    def score(self, scorer, with_sizes=True):
        """Results (and |A|, |C|, |T| unless with_sizes is False, which takes
        the kernel's path that does not count the sets)."""
        import paper_2609_33224_amd as ps
        import torch
        scorer.score_dev(self.d_pool, self.pool_len, self.d_reqs, self.n_req, self.d_out,
                         self.d_sizes if with_sizes else None)
        torch.cuda.synchronize()
        res = ps.results_from_device(self.d_out)[:self.n_req]
        if not with_sizes:
            return res, None
        sizes = self.d_sizes.cpu().numpy().view(np.uint32).reshape(-1, 3)[:self.n_req]
        return res, sizes

    def hits(self, scorer, n_inst):
        import torch
        d_hits = torch.zeros(max(self.n_req, 1) * n_inst, dtype=torch.int32, device="cuda")
        scorer.hits_dev(self.d_pool, self.pool_len, self.d_reqs, self.n_req, d_hits)
        torch.cuda.synchronize()
        return d_hits.cpu().numpy().view(np.uint32).reshape(-1, n_inst)[:self.n_req]


def compare_decisions(res, sizes, od, idx=None, tol=NB_TOL, label=""):
    """GPU results vs oracle decisions (optionally the oracle holds only the
    requests `idx` of the GPU window).  Returns the near-boundary count.
    Bit-exact on chosen instance, hit, flags and set sizes except where the
    oracle flags a near-boundary comparison; latencies within `tol`."""
    if idx is not None:
        res, sizes = res[idx], sizes[idx]
    nb_dec = (od.nb & oracle.NB_DECISION) != 0
    nb_flag = (od.nb & oracle.NB_MISSFLAG) != 0
    ok = ~nb_dec
    bad = np.nonzero(ok & ((res["instance"] != od.inst) | (res["hit_blocks"] != od.hit)))[0]
    assert len(bad) == 0, (
        f"{label}: {len(bad)} decisions differ, first r={bad[0]}: gpu "
        f"{res[bad[0]]} oracle inst={od.inst[bad[0]]} hit={od.hit[bad[0]]} "
        f"flags={od.flags[bad[0]]} sizes={od.sizes[bad[0]]} gpu sizes={sizes[bad[0]]}")
    fl_mask = np.where(nb_flag, ~np.uint32(oracle.R_TTFT_MISS), np.uint32(0xFFFFFFFF))
    fbad = np.nonzero(ok & ((res["flags"] & fl_mask) != (od.flags & fl_mask)))[0]
    assert len(fbad) == 0, f"{label}: flags differ at r={fbad[:5]}"
    sbad = np.nonzero(ok & (sizes != od.sizes).any(axis=1))[0]
    assert len(sbad) == 0, f"{label}: set sizes differ at r={sbad[:5]}: {sizes[sbad[0]]} vs {od.sizes[sbad[0]]}"
    chosen = ok & (od.inst >= 0)
    for name, ref in (("ttft", od.ttft), ("tpot", od.tpot)):
        g = res[name][chosen].astype(np.float64)
        r = ref[chosen]
        rel = np.abs(g - r) / np.maximum(np.abs(r), 1e-30)
        assert (rel <= tol).all(), f"{label}: {name} rel err {rel.max():.3g} > {tol}"
    return int(nb_dec.sum())
