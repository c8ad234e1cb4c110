"""Benchmark of the PackServe window scorer on one MI355X.

A step is one call of ps_score_window_dev over the whole window (prefix
match, latency model, filters and selection for every request x instance
pair), inputs resident in HBM.  Default workload: the 64-instance x 16,384-
request window with a 30 ms TPOT target (c2).  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload c2] [--no-cpu-baseline]

The roofline block is the scoring pass's (lean + general kernels):
algorithmic bytes from `score_bytes` over the library's HIP-event time on
the launch stream.  The probe_kernel block is the exhaustive probe kernel's
(ps_probe_hits_dev): one 64-byte bucket per probe, min(hit + 1, chain
length) probes per (request, instance) pair, plus the staged chain head;
its measured_bytes are the HBM-side bytes of its dispatches per window
(rocprofv3 FETCH_SIZE and WRITE_SIZE, scaled as for `traffic`), below the
algorithmic bytes where requests that share a segment hit in the caches.
`traffic` and measured_bytes come from the committed rocprofv3 counter
summary of the same kernel sources, or are null.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("request×instance candidate evals/sec + decisions/sec; "
          "probe-kernel % of HBM peak")
HBM_PEAK_GBS = 8000.0
BUCKET_BYTES = 64  # one 8-slot bucket of a per-instance table
PROBE_ROWPOS = BUCKET_BYTES + 4  # a probe that also reads the found slot's row position
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")

WORKLOAD_NAMES = {
    "c1": "16 instances x 1,024 requests, TPOT 50 ms",
    "c2": "64 instances x 16,384 requests, session prefixes 512-4,096 blocks, owner Zipf(1.1), TPOT 30 ms",
    "c2_50": "64 instances x 16,384 requests, session prefixes 512-4,096 blocks, owner Zipf(1.1), TPOT 50 ms",
    "c3": "1,024 instances x 65,536 requests, 40% share a 128-block system prompt, TPOT 30 ms",
    "c4": "256 instances x 32,768 requests, prefixes 2,048-12,500 blocks, 85% saturated, TPOT 50 ms",
    "c5": "4,096 instances x 262,144 requests, uniform scatter, TPOT 30 ms",
}


def kernel_source_hash() -> str:
    """Hash of the window kernel's sources (kernels, shared device helpers,
    device layout); the committed counter summary applies only to it."""
    h = hashlib.sha256()
    for name in ("ps_kernels.hip", "ps_common.h", "ps_device.h"):
        with open(os.path.join(ROOT, "paper_2609_33224_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _fp64_model(win):
    """fp64 copies of the model for byte accounting (not for decisions)."""
    import numpy as np
    a = win.alpha.astype(np.float64)
    ub = win.seg_ub.astype(np.int64)
    beta = win.beta.astype(np.float64)
    gam = win.gamma.astype(np.float64)
    return a, ub, beta, gam


def _tpf(a, n, c):
    return a[0] + a[1] * n + a[2] * n * c + a[3] * n * n + a[4] * c + a[5] * c * c


def probe_bytes(win, hits):
    """Algorithmic bytes of the exhaustive probe kernel (ps_probe_hits_dev):
    one 64-byte bucket per probe, min(hit + 1, chain length) probes on every
    (request, instance) pair, plus the chain head it stages."""
    import numpy as np
    ell = (win.pre_len.astype(np.int64) + win.tail_len)[: hits.shape[0]]
    probes = np.minimum(hits.astype(np.int64) + 1, ell[:, None])
    probes = np.where(ell[:, None] == 0, 0, probes)
    n_probes = int(probes.sum())
    return n_probes * BUCKET_BYTES + int(np.minimum(ell, 256).sum()) * 8, n_probes


GROUP_MIN, GROUP_HOLD = 8, 16  # shortest grouped segment; holders a group record keeps


def group_info(win):
    """Prefix groups as the kernels form them: requests with a shared
    segment of at least GROUP_MIN blocks and equal pre_off; per group the
    longest member segment and the first request holding it."""
    import numpy as np
    R = win.n_req
    grouped = win.pre_len >= GROUP_MIN
    idx = np.nonzero(grouped)[0]
    order = idx[np.lexsort((idx, -win.pre_len[idx].astype(np.int64), win.pre_off[idx]))]
    first = np.ones(len(order), bool)
    first[1:] = win.pre_off[order[1:]] != win.pre_off[order[:-1]]
    gid_sorted = np.cumsum(first) - 1
    gid = np.full(R, -1, np.int64)
    gid[order] = gid_sorted
    rep = order[first]
    return gid, rep, win.pre_len[rep].astype(np.int64)


def group_segment_hits(sc, win, d_pool, rep, plen, chunk_pairs=1 << 25):
    """Hit of each group's longest segment on every instance (the walk the
    group pass makes), from the exhaustive hits of the representatives."""
    import numpy as np
    import torch
    import paper_2609_33224_amd as ps
    G, N = len(rep), win.n_inst
    H = np.zeros((G, N), np.int64)
    if G == 0:
        return H
    reqs = ps.pack_reqs(win.pre_off[rep], win.pre_len[rep], win.tail_off[rep], win.tail_len[rep])
    chunk = max(1, min(G, chunk_pairs // N))
    d_hits = torch.empty(chunk * N, dtype=torch.int32, device="cuda")
    for g0 in range(0, G, chunk):
        n = min(chunk, G - g0)
        sc.hits_dev(d_pool, len(win.pool), ps.to_device_bytes(reqs[g0:g0 + n]), n, d_hits)
        torch.cuda.synchronize()
        h = d_hits[: n * N].cpu().numpy().view(np.uint32).reshape(n, N).astype(np.int64)
        H[g0:g0 + n] = np.minimum(h, plen[g0:g0 + n, None])
    return H


def index_walk_bytes(h, ell, nw, h_all=None):
    """Bytes of walking the live holders (h >= 1) of a chain of ell blocks
    together through the prefix index: per position up to the second
    longest hit one 128-byte index bucket plus that position's holders in
    the pool (hits h_all, default h; a 2-byte id each, or the bitmap's
    8-byte words for more than 64 holders), then the longest holder alone
    along its row."""
    import numpy as np
    if h_all is None:
        h_all = h
    hr = np.sort(h[h >= 1])[::-1]
    if len(hr) == 0 or ell <= 1:
        return 0
    P = int(min(ell - 1, hr[1] if len(hr) > 1 else 0))
    by = 0
    if P > 0:
        cnts = (h_all[None, :] > np.arange(1, P + 1)[:, None]).sum(1)
        by += 128 * P + int(np.where(cnts > 64, 8 * nw, 2 * cnts).sum())
    if hr[0] > P:
        by += PROBE_ROWPOS + 16 * max(0, min(int(hr[0]), ell - 1) - (P + 1)) + (BUCKET_BYTES if hr[0] < ell else 0)
    return by


def group_classes(H):
    """The shared-hit class of each group as the group kernel forms it (for
    popular groups with more than 64 holders of the first block): H* = the
    most frequent hit among the holders in the first 64-instance word that
    has any (the lowest-lane value among equally frequent ones), the
    exceptions = the holders whose hit differs; class-able with at most
    GROUP_HOLD exceptions.  Returns (classable, H*, exception mask)."""
    import numpy as np
    G, N = H.shape
    ok = np.zeros(G, bool)
    hs = np.zeros(G, np.int64)
    exc = np.zeros((G, N), bool)
    hold = H >= 1
    for k in np.nonzero(hold.sum(1) > 64)[0]:
        w = int(np.argmax(hold[k].reshape(-1, 64).any(1))) if N % 64 == 0 else None
        if w is None:
            words = [hold[k][i:i + 64] for i in range(0, N, 64)]
            w = next(i for i, x in enumerate(words) if x.any())
        lanes = np.nonzero(hold[k][w * 64:(w + 1) * 64])[0]
        vals = H[k][w * 64 + lanes]
        best, bestc = 0, 0
        seen = set()
        for v in vals:  # distinct values in lane order; a strictly larger count wins
            if v in seen:
                continue
            seen.add(v)
            c = int((vals == v).sum())
            if c > bestc:
                best, bestc = int(v), c
        hs[k] = best
        exc[k] = hold[k] & (H[k] != best)
        ok[k] = exc[k].sum() <= GROUP_HOLD and 0 < best < (1 << 24)
    return ok, hs, exc


def group_pass_bytes(win, gid, rep, plen, H):
    """Algorithmic bytes of the prefix-group pass.  Claim: descriptor, slot
    read, the claiming compare-and-swap, the length maximum and the slot
    entry per request.  Walk: slot entry per request; per group its
    segment head staged (<= 256 hashes), one index bucket, the holder ids
    (or bitmap), then with at most GROUP_HOLD holders per holder a probe of
    the first block with its row position, 16 bytes per compared position,
    a final probe where the segment leaves the cache, and the record; with
    more, the holders walked together through the index and one 4-byte hit
    per holder in the popular row, and for more than 64 holders the bitmap
    and the hits read back for the shared-hit class, and its word."""
    import numpy as np
    R, N = win.n_req, win.n_inst
    nw = (N + 63) // 64
    g = gid >= 0
    by = 28 * R + int(g.sum()) * (8 + 16) + len(rep) * 16
    by += 4 * R
    cnt0 = (H >= 1).sum(1)
    by += int((16 + 8 * np.minimum(plen, 256) + 128 +
               np.where(cnt0 > 64, 8 * nw, 2 * cnt0)).sum())
    ok = cnt0 <= GROUP_HOLD
    hc = np.minimum(H, (plen - 1)[:, None])
    walk = np.where(H >= 1, PROBE_ROWPOS + 16 * hc + BUCKET_BYTES * (H < plen[:, None]), 0)
    walk = np.where((plen > 1)[:, None], walk, np.where(H >= 1, PROBE_ROWPOS, 0))
    by += int(walk[ok].sum()) + int((8 + 8 * cnt0[ok]).sum())
    for k in np.nonzero(~ok)[0]:
        by += 8 + index_walk_bytes(H[k], int(plen[k]), nw) + 4 * int(cnt0[k])
        if cnt0[k] > 64:  # the shared-hit class: bitmap and hits read back, the class word
            by += 8 * nw + 4 * int(cnt0[k]) + 8
    return by


def score_bytes(win, r0, hits, grp=None):
    """Algorithmic bytes the scoring pass moves for requests r0 .. r0 +
    len(hits) (the benchmark's policy: D-C-Q, monotone model, no set sizes).

    Requests whose group record holds their hits go through the lean kernel
    (four requests per wave): 24 B descriptor + 4 B group slot + 136 B
    record + 20 B result; for pools above 64 instances 32 B of state per
    holder of the first block (that read also decides eligibility), 64 x
    16 B per chunk of zero-hit thresholds read (the first chunk that admits
    the request's length is read in any case, later ones until an admitted
    non-holder is found) and 32 B for the chosen instance's state when an
    admitted non-holder is found (an upper bound: it is read only when that
    instance wins); a resume walk on each candidate whose shared segment is
    cached to the request's segment end (a probe with its row position, 16
    B per compared position, a final probe); when no member of the hit-0
    class and no candidate is in T, the states of all instances.  Pools of
    at most 64 instances keep states and thresholds in LDS (no bytes).  The
    rooms and threshold maxima are read once per wave (not counted).

    Requests of a popular group with a shared-hit class below their
    segment end take the general kernel's class path: descriptor, slot,
    144 B record, result, the 64 largest rooms (1 KB), the holder bitmap,
    32 B per exception's state and its resume walk, the 16-byte summaries
    of the key-ordered chunks, one chunk of 64 key-ordered states with
    their ids, one chunk of thresholds with the chunk maxima, and the
    chosen state (a lower bound: later chunks and the fallback scan are
    not counted).

    Other requests go through the general kernel: descriptor, slot, result;
    the 64-way search of the sorted rooms; with a popular group row the
    record, one 128-byte index bucket, the first block's holders (2-byte ids
    + 8-byte rooms, or the bitmap's words + rooms) and a 4-byte hit per
    candidate; without a group the staged chain head and the per-request
    walks (per walked holder a probe with its row position, 16 B per
    compared position and a final probe; with more than 64 holders the
    index walk); 32 B of state per member of C; the zero-hit threshold
    search (4 B per chunk maximum, 16 B per threshold of each visited chunk)
    or, when the class must be evaluated, 8 B room + 32 B state per eligible
    non-holder."""
    import numpy as np
    R, N = hits.shape
    pol = win.policy
    bs, bmax, kv = int(pol["block_tokens"]), int(pol["b_max"]), int(pol["kv_cap_tokens"])
    eta, tau = float(np.float32(pol["eta"])), float(np.float32(pol["tpot_slo"]))
    lout1 = max(1.0, float(np.float32(pol["lout"])))
    a, ub, beta, gam = _fp64_model(win)
    sl = slice(r0, r0 + R)
    ell = win.pre_len[sl].astype(np.int64) + win.tail_len[sl]
    p = win.pre_len[sl].astype(np.int64)
    L = ell * bs
    A1 = win.D.astype(np.int64) + win.Q + 1
    room = np.where(A1 <= bmax, kv - win.S, -1)
    small = N <= 64
    nw = (N + 63) // 64
    n1 = nw
    levels, span = 1, N
    while span > 64:
        span = (span + 63) // 64
        levels += 1
    h = hits.astype(np.int64)
    elig = room[None, :] >= L[:, None]
    hold0 = h >= 1
    cand = elig & hold0
    ncand = cand.sum(1)
    nA = elig.sum(1)
    cnt0 = hold0.sum(1)
    act = nA > 0
    if grp is None:
        grp = dict(has=np.zeros(R, bool), pop=np.zeros(R, bool), grouped=np.zeros(R, bool),
                   Hg=np.zeros_like(h))
    lean = grp["has"] & ~grp["pop"]
    pop = grp["has"] & grp["pop"]
    # popular groups with a shared-hit class, where H* lies below the
    # request's segment end (p0): the class path of the general kernel
    if "cls" in grp:
        p0 = np.minimum(win.pre_len[r0:r0 + R].astype(np.int64), grp["gplen"])
        clsp = grp["cls"] & (grp["hs"] < p0)
    else:
        clsp = np.zeros(R, bool)
    pop = pop & ~clsp
    # resume walks of grouped requests
    Hg = grp["Hg"]
    resume = cand & (Hg >= p[:, None]) & (p < ell)[:, None]
    rb = np.where(h > p[:, None],
                  PROBE_ROWPOS + 16 * (np.minimum(h, (ell - 1)[:, None]) - p[:, None]) +
                  BUCKET_BYTES * (h < ell[:, None]), PROBE_ROWPOS)
    resume_by = np.where(resume, rb, 0).sum(1)
    # general kernel: per-request parts
    gen = 48 + 512 * levels + np.zeros(R, np.int64)
    gen += np.where(pop, 144 + np.where(act & (ell > 0), 128 + np.where(
        cnt0 <= 64, 10 * cnt0, 8 * nw + 8 * cnt0) + 4 * ncand, 0) + resume_by, 0)
    nogrp = ~grp["has"]
    gen += np.where(nogrp, 8 * np.minimum(ell, 256) + np.where(grp["grouped"], 144, 0), 0)
    gen += np.where(nogrp & act & (ell > 0), 128 + np.where(cnt0 <= 64, 10 * cnt0, 8 * nw + 8 * cnt0), 0)
    few = ncand <= 64
    hc = np.minimum(h, (ell - 1)[:, None])
    walk = np.where(cand, PROBE_ROWPOS + 16 * hc + BUCKET_BYTES * (h < ell[:, None]), 0).sum(1)
    gen += np.where(nogrp & act & few & (ell > 1), walk, 0)
    for r in np.nonzero(nogrp & act & ~few & (ell > 1))[0]:
        gen[r] += index_walk_bytes(np.where(cand[r], h[r], 0), int(ell[r]), nw, h[r])
    # lean kernel: per-request parts
    lby = 184 + (0 if small else 32) * cnt0 + resume_by
    lby = np.where(act, lby, 184)
    by = np.where(lean, lby, gen)
    if clsp.any():
        exc = grp["exc"]
        ex_res = np.where(resume & exc, rb, 0).sum(1)
        cby = (24 + 4 + 8 * 18 + 20 + 64 * 16 + 8 * nw + 32 * exc.sum(1) + ex_res +
               16 * n1 + 64 * (4 + 32) + 4 * n1 + 64 * 16 + 32)
        by = np.where(clsp, cby, by)
    # the recomputation filter and the hit-0 class
    n = (L[:, None] - h * bs).astype(np.float64)
    c = (h * bs).astype(np.float64)
    Lf = L.astype(np.float64)[:, None]
    W = np.maximum(0.0, _tpf(a, n, c) - _tpf(a, 0.0, Lf))
    Z = (_tpf(a, Lf, 0.0) - _tpf(a, 0.0, Lf))[:, 0]
    Wmin = np.where(elig, W, np.inf).min(1)
    kvc = Z > 0
    with np.errstate(divide="ignore", invalid="ignore"):
        rho = (W - Wmin[:, None]) / Z[:, None]
    inC = elig & (~kvc[:, None] | (rho <= eta))
    by += np.where(lean | clsp, 0, 32 * (cand & inC).sum(1))
    n0 = nA - ncand
    W0 = np.maximum(0.0, Z)
    with np.errstate(divide="ignore", invalid="ignore"):
        admit0 = (n0 > 0) & (~kvc | ((W0 - Wmin) / Z <= eta))
    seg = np.searchsorted(ub, A1, side="left")
    seg = np.minimum(seg, len(ub) - 1)
    order0 = np.lexsort((np.arange(N), win.Q, -win.D.astype(np.int64)))
    chunk_lean = 0 if small else 64 * 16
    for r in np.nonzero(act & (admit0 | lean) & ~clsp)[0]:
        t_iter = gam[seg] * (beta[seg, 0] + beta[seg, 1] * A1 + beta[seg, 2] * (win.S + L[r]))
        tpot0 = t_iter + np.where(A1 > 1, _tpf(a, float(L[r]), 0.0) / lout1, 0.0)
        zero = elig[r] & ~hold0[r]
        feas = np.zeros(n1 * 64, bool)
        feas[:N] = (elig[r] & (tpot0 < tau))[order0]
        passing = feas.reshape(n1, 64).any(1)
        ok = (zero & (tpot0 < tau))[order0]
        found = bool(ok.any())
        cs = int(np.argmax(ok)) // 64 if found else n1 - 1
        if lean[r]:
            if not admit0[r]:  # only the speculative first chunk
                by[r] += chunk_lean if passing.any() else 0
                continue
            by[r] += chunk_lean * int(passing[:cs + 1].sum()) + (0 if small or not found else 32)
        else:
            by[r] += 256 * (cs // 64 + 1) + 1024 * int(passing[:cs + 1].sum())
        if found:
            continue
        # No member of the class is in T: it is evaluated in full only when
        # no candidate is in T either.
        cr = cand[r] & inC[r]
        if cr.any():
            tp = t_iter[cr] + np.where(A1[cr] > 1, _tpf(a, n[r][cr], c[r][cr]) / lout1, 0.0)
            if (tp < tau).any():
                continue
        if lean[r]:
            by[r] += 0 if small else 32 * N + 32
        else:
            by[r] += 8 * N + 32 * int(zero.sum())
    return int(by.sum())


def algorithmic_bytes(sc, win, d_pool, d_reqs, chunk_pairs=1 << 25):
    """The byte counts of the scoring kernel, the prefix-group pass and the
    exhaustive probe kernel over the whole window, from the exhaustive
    per-pair hits exported chunk by chunk (untimed)."""
    import numpy as np
    import torch
    import paper_2609_33224_amd as ps
    gid, rep, plen = group_info(win)
    H = group_segment_hits(sc, win, d_pool, rep, plen)
    # every group gets a result: a record, or a popular row (the area holds
    # 64 MiB / (4 n_inst) rows, more than any benchmark window needs)
    g_has = np.ones(len(rep), bool)
    g_pop = (H >= 1).sum(1) > GROUP_HOLD if len(rep) else np.zeros(0, bool)
    assert int(g_pop.sum()) <= (64 << 20) // (4 * win.n_inst)
    gb = group_pass_bytes(win, gid, rep, plen, H)
    g_cls, g_hs, g_exc = group_classes(H) if len(rep) else (np.zeros(0, bool), np.zeros(0, np.int64),
                                                            np.zeros((0, win.n_inst), bool))
    chunk = max(1, min(win.n_req, chunk_pairs // win.n_inst))
    reqs = ps.pack_reqs(win.pre_off, win.pre_len, win.tail_off, win.tail_len)
    d_hits = torch.empty(chunk * win.n_inst, dtype=torch.int32, device="cuda")
    sb = pb = npr = 0
    for r0 in range(0, win.n_req, chunk):
        n = min(chunk, win.n_req - r0)
        d_r = ps.to_device_bytes(reqs[r0:r0 + n])
        sc.hits_dev(d_pool, len(win.pool), d_r, n, d_hits)
        torch.cuda.synchronize()
        hits = d_hits[: n * win.n_inst].cpu().numpy().view(np.uint32).reshape(n, win.n_inst)
        b, p_ = probe_bytes(win.subset(range(r0, r0 + n)), hits)
        pb += b
        npr += p_
        gc = gid[r0:r0 + n]
        grouped = gc >= 0
        has = grouped & g_has[np.maximum(gc, 0)] if len(rep) else grouped
        pop = grouped & g_pop[np.maximum(gc, 0)] if len(rep) else grouped
        Hg = H[np.maximum(gc, 0)] if len(rep) else np.zeros(hits.shape, np.int64)
        gi = np.maximum(gc, 0)
        cls = pop & g_cls[gi] if len(rep) else np.zeros(n, bool)
        hs = g_hs[gi] if len(rep) else np.zeros(n, np.int64)
        exc = g_exc[gi] if len(rep) else np.zeros(hits.shape, bool)
        gpl = plen[gi] if len(rep) else np.zeros(n, np.int64)
        sb += score_bytes(win, r0, hits, dict(has=has, pop=pop, grouped=grouped, Hg=Hg, cls=cls,
                                              hs=hs, exc=exc, gplen=gpl))
    return sb, gb, pb, npr


def traffic_for(workload: str, src_hash: str):
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    ent = t.get(workload)
    if not ent or ent.get("kernel_source_sha") != src_hash:
        return None
    return ent


def cpu_baseline(win, budget_s: float):
    """The oracle on the host cores, over the same window, repeated (or on a
    leading slice) to fill roughly `budget_s` seconds."""
    import oracle
    o = oracle.Oracle.from_window(win)
    threads = oracle.max_threads()
    t0 = time.perf_counter()
    o.window_score(win)
    one = time.perf_counter() - t0
    if one > budget_s:
        n = max(64, int(win.n_req * budget_s / one))
        sub = win.subset(range(n))
        t0 = time.perf_counter()
        o.window_score(sub)
        dt = time.perf_counter() - t0
        return dict(value=n * win.n_inst / dt, unit="candidate evals/s", cores=threads,
                    kind="oracle", decisions_per_s=n / dt,
                    sample=f"first {n} of {win.n_req} requests of the window, once")
    reps = max(1, int(budget_s / max(one, 1e-3)))
    t0 = time.perf_counter()
    for _ in range(reps):
        o.window_score(win)
    dt = (time.perf_counter() - t0) / reps
    return dict(value=win.n_req * win.n_inst / dt, unit="candidate evals/s", cores=threads,
                kind="oracle", decisions_per_s=win.n_req / dt,
                sample=f"whole window ({win.n_req} requests x {win.n_inst} instances), "
                       f"{reps} repetitions")


def cpu_sequential_baseline(win, budget_s: float):
    """The oracle's Algorithm 1 per arrival (one thread: each request waits
    for the one before it) over the window or its leading slice."""
    import oracle
    o = oracle.Oracle.from_window(win)
    n = win.n_req
    t0 = time.perf_counter()
    o.window_schedule(win.subset(range(min(n, 256))))
    one = (time.perf_counter() - t0) / min(n, 256)
    if one * n > budget_s:
        n = max(256, int(budget_s / max(one, 1e-9)))
    o = oracle.Oracle.from_window(win)
    t0 = time.perf_counter()
    o.window_schedule(win.subset(range(n)) if n < win.n_req else win)
    dt = time.perf_counter() - t0
    return dict(value=n / dt, unit="decisions/s", cores=1, kind="oracle",
                sample=(f"first {n} of {win.n_req} requests, per arrival, once" if n < win.n_req
                        else f"whole window ({win.n_req} requests), per arrival, once"))


def sequential_block(sc, win, model, d_pool, d_reqs, snap, reps, stream):
    """Algorithm 1 per arrival (ps_schedule_window_dev) on the same window and
    starting state, and the herding of the snapshot placements: the same
    placements replayed in arrival order (ps_replay_window_dev)."""
    import numpy as np
    import torch
    import paper_2609_33224_amd as ps

    def reload():
        sc.load(win.n_inst, win.cap, win.blk_off, win.blk, win.D, win.Q, win.P, win.S, model)
        torch.cuda.synchronize()

    n = win.n_req
    snap_all = snap
    d_out = torch.empty(n * 20, dtype=torch.uint8, device="cuda")
    times = []
    for k in range(reps + 1):  # the first call is a warm-up
        reload()
        t0 = time.perf_counter()
        sc.schedule_dev(d_pool, len(win.pool), d_reqs, n, d_out, None, stream)
        dt = time.perf_counter() - t0
        if k:
            times.append(dt)
    seq = ps.results_from_device(d_out)
    # The replay stops before the first placement that would take an
    # instance's queue past its 12-bit limit (snapshot herding can).
    n_rep, q = n, win.Q.astype(np.int64).copy()
    for k, i in enumerate(snap["instance"]):
        if i >= 0:
            q[i] += 1
            if q[i] > 4095:
                n_rep = k
                break
    reload()
    d_inst = torch.from_numpy(np.ascontiguousarray(snap["instance"][:n_rep], np.int32)).to("cuda")
    t0 = time.perf_counter()
    if n_rep:
        sc.replay_dev(d_pool, len(win.pool), d_reqs, n_rep, d_inst, d_out, stream)
    replay_s = time.perf_counter() - t0
    rep = ps.results_from_device(d_out)[:n_rep]
    snap = snap[:n_rep]
    tau = float(np.float32(win.policy["tpot_slo"]))
    fb = ps.PS_R_FALLBACK
    ok_snap = (snap["instance"] >= 0) & ((snap["flags"] & fb) == 0)
    ok_seq = (seq["instance"] >= 0) & ((seq["flags"] & fb) == 0)
    per_snap = np.bincount(snap_all["instance"][snap_all["instance"] >= 0], minlength=win.n_inst)
    per_seq = np.bincount(seq["instance"][seq["instance"] >= 0], minlength=win.n_inst)
    ms = float(np.mean(times)) * 1e3
    return {
        "entry": "ps_schedule_window_dev: Algorithm 1 per arrival (hits pass, one-workgroup "
                 "scheduler, rebuild of the derived data)",
        "ms_per_window": ms, "decisions_per_s": n / (ms * 1e-3),
        "us_per_decision": ms * 1e3 / n, "reps": reps,
        "bound": "latency (each decision waits for the commit before it)",
        "placed": int((seq["instance"] >= 0).sum()),
        "fallback": int(((seq["flags"] & fb) != 0).sum()),
        "tpot_at_or_above_target_non_fallback": int((seq["tpot"][ok_seq] >= tau).sum()),
        "herding": {
            "snapshot_choice_differs_frac": float(np.mean(seq["instance"] != snap_all["instance"])),
            "replayed_requests": int(n_rep),
            "snapshot_non_fallback_placed": int(ok_snap.sum()),
            "snapshot_tpot_at_or_above_target_at_arrival": int((rep["tpot"][ok_snap] >= tau).sum()),
            "snapshot_ttft_miss_at_arrival": int(((rep["flags"] & ps.PS_R_TTFT_MISS) != 0).sum()),
            "max_requests_per_instance": {"snapshot": int(per_snap.max()),
                                          "per_arrival": int(per_seq.max())},
            "replay_ms": replay_s * 1e3,
        },
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c2", choices=sorted(WORKLOAD_NAMES))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--sequential-reps", type=int, default=3,
                    help="timed calls of the per-arrival scheduler (0: skip that block)")
    ap.add_argument("--skip-bytes", action="store_true",
                    help="skip the algorithmic byte counts (roofline fields null; for counter runs)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run 5 device-to-device copies of this many MiB (a plain copy "
                         "kernel of known size, to scale the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the request-sharded multi-GPU design is described in DESIGN.md)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 20
        src = torch.ones(n // 8, dtype=torch.int64, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "copies": 5}))
        return
    import synth
    import paper_2609_33224_amd as ps

    print(f"bench: generating {args.workload}", file=sys.stderr, flush=True)
    win = synth.generate(args.workload, seed=args.seed)
    sc = ps.Scorer(0)
    m = ps.make_model(win.alpha, win.seg_ub, win.beta, win.gamma, win.policy["eta"],
                      win.policy["tpot_slo"], win.policy["ttft_floor"], win.policy["lout"],
                      win.policy["block_tokens"], win.policy["b_max"],
                      win.policy["kv_cap_tokens"], win.policy["flags"], win.policy["rand_seed"])
    t0 = time.perf_counter()
    sc.load(win.n_inst, win.cap, win.blk_off, win.blk, win.D, win.Q, win.P, win.S, m)
    load_s = time.perf_counter() - t0
    reqs = ps.pack_reqs(win.pre_off, win.pre_len, win.tail_off, win.tail_len)
    d_pool = ps.to_device_u64(win.pool)
    d_reqs = ps.to_device_bytes(reqs)
    d_out = torch.empty(win.n_req * 20, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    # untimed: byte counts from the per-pair hits, and the end-to-end host call
    if args.skip_bytes:
        alg_bytes = group_bytes = probe_alg_bytes = n_probes = None
    else:
        print("bench: counting algorithmic bytes", file=sys.stderr, flush=True)
        alg_bytes, group_bytes, probe_alg_bytes, n_probes = algorithmic_bytes(sc, win, d_pool, d_reqs)
    t0 = time.perf_counter()
    sc.score(win.pool, reqs)
    host_call_s = time.perf_counter() - t0

    # the exhaustive per-instance probe kernel (ps_probe_hits_dev), timed alone
    pk_chunk = max(1, min(win.n_req, (1 << 28) // win.n_inst))
    d_ph = torch.empty(pk_chunk * win.n_inst, dtype=torch.int32, device="cuda")
    d_pr = ps.to_device_bytes(reqs[:pk_chunk])
    sc.hits_dev(d_pool, len(win.pool), d_pr, pk_chunk, d_ph, stream)
    pe = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(3)]
    for a_, b_ in pe:
        a_.record(stream)
        sc.hits_dev(d_pool, len(win.pool), d_pr, pk_chunk, d_ph, stream)
        b_.record(stream)
    torch.cuda.synchronize()
    probe_ms = float(np.mean([a_.elapsed_time(b_) for a_, b_ in pe])) * win.n_req / pk_chunk
    del d_ph, d_pr

    for _ in range(args.warmup):
        sc.score_dev(d_pool, len(win.pool), d_reqs, win.n_req, d_out, None, stream)
    torch.cuda.synchronize()
    # The timed region: exactly K steps back to back, bracketed by device
    # synchronisation (no events inside it: a marker between steps costs the
    # stream a few microseconds of its own).
    print(f"bench: timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for _ in range(args.steps):
        sc.score_dev(d_pool, len(win.pool), d_reqs, win.n_req, d_out, None, stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_per_step = wall * 1e3 / args.steps
    res = ps.results_from_device(d_out)
    # The same steps again, each between two events (per-step device time).
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        a.record(stream)
        sc.score_dev(d_pool, len(win.pool), d_reqs, win.n_req, d_out, None, stream)
        b.record(stream)
    torch.cuda.synchronize()
    step_avg = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    # The same steps again with the library's events around its launches:
    # the prefix-group pass and the scoring kernel, each on the launch stream.
    sc.set_timing(True)
    for _ in range(args.steps):
        sc.score_dev(d_pool, len(win.pool), d_reqs, win.n_req, d_out, None, stream)
    n_timed, group_ms, kern_avg = sc.read_timing()
    sc.set_timing(False)

    evals = win.n_req * win.n_inst
    src_hash = kernel_source_hash()
    from paper_2609_33224_amd import build as ps_build
    lib_id = ps.ps_build_id()
    lib_fresh = lib_id == ps_build.source_hash()
    if not lib_fresh:
        print(f"bench: libpackserve.so was built from other sources ({lib_id}); "
              "rebuild it (__graft_entry__.build()); counter bytes are not applied", file=sys.stderr)
    tent = (traffic_for(args.workload, src_hash) or {}) if lib_fresh else {}
    traffic = tent.get("bytes_per_launch")
    probe_meas = tent.get("probe_bytes_per_window")
    def rate(nbytes, ms):
        return nbytes / (ms * 1e-3) / 1e9 if nbytes is not None and ms > 0 else None

    achieved = rate(alg_bytes, kern_avg)
    probe_gbs = rate(probe_alg_bytes, probe_ms)
    out = {
        "metric": METRIC,
        "value": evals / (ms_per_step * 1e-3),
        "unit": "candidate evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {WORKLOAD_NAMES[args.workload]}",
                   "n_inst": win.n_inst, "n_req": win.n_req, "seed": args.seed},
        "decisions_per_s": win.n_req / (ms_per_step * 1e-3),
        "step_ms_events": step_avg,
        "kernel": "scoring pass: lean_rows_kernel (four requests per wave) + general score_kernel (prefix hits from the group records, latency model, filters, keys)",
        "kernel_ms_avg": kern_avg,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS if achieved is not None else None,
                     "traffic": traffic},
        "algorithmic_bytes_per_launch": alg_bytes,
        "group_pass": {"kernels": "group_claim_kernel + group_kernel (walk of each shared "
                                  "segment once per window)",
                       "ms_avg": group_ms, "algorithmic_bytes": group_bytes,
                       "achieved_GBs": rate(group_bytes, group_ms),
                       "groups": int(len(np.unique(win.pre_off[win.pre_len >= GROUP_MIN]))),
                       "timed_calls": n_timed},
        "probe_kernel": {"kernel": "ps_probe_hits_dev (every request x instance probed)",
                         "ms_per_window": probe_ms, "probes": n_probes,
                         "algorithmic_bytes": probe_alg_bytes,
                         "achieved_GBs": probe_gbs,
                         "frac_of_hbm_peak": probe_gbs / HBM_PEAK_GBS if probe_gbs is not None else None,
                         "measured_bytes": probe_meas,
                         "measured_GBs": rate(probe_meas, probe_ms),
                         "measured_frac_of_hbm_peak": (rate(probe_meas, probe_ms) / HBM_PEAK_GBS
                                                       if probe_meas is not None else None),
                         "evals_per_s": win.n_req * win.n_inst / (probe_ms * 1e-3)},
        "kernel_source_sha": src_hash,
        "library_build_id": lib_id,
        "library_matches_sources": lib_fresh,
        "load_instances_s": load_s,
        "host_call_s_incl_pcie": host_call_s,
        "placed": int((res["instance"] >= 0).sum()),
        "fallback": int(((res["flags"] & ps.PS_R_FALLBACK) != 0).sum()),
    }
    if args.sequential_reps > 0:
        print("bench: per-arrival scheduling", file=sys.stderr, flush=True)
        out["sequential"] = sequential_block(sc, win, m, d_pool, d_reqs, res,
                                             args.sequential_reps, stream)
    sc.close()
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(win, args.cpu_budget)
        if args.sequential_reps > 0:
            out["cpu_baseline"]["sequential"] = cpu_sequential_baseline(win, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
