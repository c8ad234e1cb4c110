"""Benchmark of the PackServe window scorer on one MI355X.

A step is one call of ps_score_window_dev over the whole window (prefix
match, latency model, filters and selection for every request x instance
pair), inputs resident in HBM.  Default workload: the largest window, 4,096
instances x 262,144 requests with a 30 ms TPOT target (c5).  Prints one JSON
line.

  python bench.py [--steps K] [--warmup W] [--workload c5] [--no-cpu-baseline]

The roofline block is the dominant kernel's (the longest of the call's four
launches): its algorithmic bytes (the byte model below, per launch) over
its mean duration from the library's HIP events on the launch stream;
`traffic` is the rocprofv3 FETCH_SIZE + WRITE_SIZE bytes of the same kernel
per dispatch, scaled by what the counters read for a plain copy, from the
committed counter summary of these kernel sources (else null).  `kernels`
gives the same for every launch of the call; `call` the whole call's bytes
over the step time; `per_pair_walk` what walking every eligible pair would
move.  The probe_kernel block is the exhaustive probe kernel's
(ps_probe_hits_dev): one 64-byte bucket per probe, min(hit + 1, chain
length) probes per (request, instance) pair, plus the staged chain head.
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
POP_WORDS = 64  # the popular pass takes pools of at most 64 x 64 instances
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


def probe_bytes(win, r0, pr, ph, n_rows, N):
    """Algorithmic bytes of the exhaustive probe kernel (ps_probe_hits_dev)
    for requests r0 .. r0 + n_rows given their holder pairs (rows pr, hits
    ph >= 1): one 64-byte bucket per probe, min(hit + 1, chain length)
    probes on every (request, instance) pair (one on a pair with hit 0 and a
    non-empty chain), plus the chain head it stages.  Returns (bytes,
    probes)."""
    import numpy as np
    ell = (win.pre_len.astype(np.int64) + win.tail_len)[r0:r0 + n_rows]
    cnt = np.bincount(pr, minlength=n_rows)
    n_probes = int(((N - cnt) * (ell > 0)).sum() + np.minimum(ph + 1, ell[pr]).sum())
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
    group pass makes), from the exhaustive hits of the representatives, as
    sorted sparse pairs: keys g * n_inst + i and hits >= 1."""
    import numpy as np
    import torch
    import paper_2609_33224_amd as ps
    G, N = len(rep), win.n_inst
    keys, vals = [np.zeros(0, np.int64)], [np.zeros(0, np.int64)]
    if G == 0:
        return keys[0], vals[0]
    reqs = ps.pack_reqs(win.pre_off[rep], win.pre_len[rep], win.tail_off[rep], win.tail_len[rep])
    chunk = max(1, min(G, chunk_pairs // N))
    d_hits = torch.empty(chunk * N, dtype=torch.int32, device="cuda")
    for g0 in range(0, G, chunk):
        n = min(chunk, G - g0)
        sc.hits_dev(d_pool, len(win.pool), ps.to_device_bytes(reqs[g0:g0 + n]), n, d_hits)
        torch.cuda.synchronize()
        h = d_hits[: n * N].cpu().numpy().view(np.uint32).reshape(n, N)
        gr, gi = np.nonzero(h)
        keys.append((gr.astype(np.int64) + g0) * N + gi)
        vals.append(np.minimum(h[gr, gi].astype(np.int64), plen[g0 + gr]))
    return np.concatenate(keys), np.concatenate(vals)


def _lookup(keys, vals, q):
    """vals at the sorted keys q (0 where absent)."""
    import numpy as np
    if len(keys) == 0:
        return np.zeros(len(q), np.int64)
    k = np.minimum(np.searchsorted(keys, q), len(keys) - 1)
    return np.where(keys[k] == q, vals[k], 0)

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


def group_classes(Hk, Hv, G, N):
    """The shared-hit class of each group as the group kernel forms it (for
    popular groups with more than 64 holders of the first block): H* = the
    most frequent hit among the holders in the first 64-instance word that
    has any (the lowest-lane value among equally frequent ones), the
    exceptions = the holders whose hit differs; class-able with at most
    GROUP_HOLD exceptions.  Hk, Hv: the sparse group hits.  Returns
    (classable, H*)."""
    import numpy as np
    ok = np.zeros(G, bool)
    hs = np.zeros(G, np.int64)
    gk = Hk // N
    cnt = np.bincount(gk, minlength=G)
    start = np.concatenate([[0], np.cumsum(cnt)])
    for k in np.nonzero(cnt > 64)[0]:
        ids = Hk[start[k]:start[k + 1]] % N          # ascending
        hv = Hv[start[k]:start[k + 1]]
        w = ids[0] // 64
        vals = hv[ids // 64 == w]                    # lane order
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
        ok[k] = int((hv != best).sum()) <= GROUP_HOLD and 0 < best < (1 << 24)
    return ok, hs

def group_pass_bytes(win, gid, rep, plen, Hk, Hv):
    """Algorithmic bytes of the prefix-group pass, as (claim pass, walk).
    Claim: descriptor, slot read, the claiming compare-and-swap, the length
    maximum and the slot entry per request, a leader-list entry per group.
    Walk: slot entry per request; per group its list entry and length, its
    first block and one index bucket, then with at most GROUP_HOLD holders
    their ids and per holder a probe of the first block with its row
    position, 16 bytes per compared position (chain and row), a final probe
    where the segment leaves the cache, and the record; with more, the
    segment head staged (<= 256 hashes), the holder ids (or bitmap), the
    holders walked together through the index and one 4-byte hit per holder
    in the popular row, and for more than 64 holders the bitmap and the hits
    read back for the shared-hit class, and its word.  On pools of at most 4,096
    instances, groups whose first block has more than 64 holders go to the
    popular pass instead (the walk pass reads their class word), listed by
    the claim pass (per leader its first
    block and index bucket, per listed group its entry, class word and
    representative minimum; counted when the window has such groups), per
    first block one walk of its representative's segment through the index
    in rounds of 128 positions until one holder is left, plus the prefix
    row; per group its staged head, 16 bytes per position of the common
    prefix with the representative's segment, the prefix row, the walk on
    from there, the hits, the class and the record.  Hk, Hv: the sparse
    group hits."""
    import numpy as np
    R, N = win.n_req, win.n_inst
    G = len(rep)
    nw = (N + 63) // 64
    g = gid >= 0
    claim = 28 * R + int(g.sum()) * (8 + 16) + G * 16
    walk = 4 * R
    gk = Hk // N
    cnt0 = np.bincount(gk, minlength=G)
    ok = cnt0 <= GROUP_HOLD
    pop_pass = N <= 64 * POP_WORDS and bool((cnt0 > 64).any())
    in_pop = (cnt0 > 64) & pop_pass
    # per group: list entry and length, first block, index bucket; then the
    # holder ids (few), the class word (popular pass), or the staged head and
    # the holder ids or bitmap (the walk pass's index walk)
    walk += int((16 + 8 + 128 + np.where(
        ok, 2 * cnt0, np.where(in_pop, 8, 8 * np.minimum(plen, 256) +
                               np.where(cnt0 > 64, 8 * nw, 2 * cnt0)))).sum())
    pl = plen[gk]
    w = np.where(pl > 1, PROBE_ROWPOS + 16 * np.minimum(Hv, pl - 1) + BUCKET_BYTES * (Hv < pl),
                 PROBE_ROWPOS)
    walk += int(w[ok[gk]].sum()) + int((8 + 8 * cnt0[ok]).sum())
    start = np.concatenate([[0], np.cumsum(cnt0)])
    popular = np.nonzero(~ok)[0]
    if pop_pass:
        # the claim pass lists the popular pass's groups: per leader its
        # first block and index bucket; per listed group its entry, class
        # word and a minimum
        claim += G * (8 + 128) + 24 * int((cnt0 > 64).sum())
    first_block = {}
    for k in popular:
        h = np.zeros(N, np.int64)
        h[Hk[start[k]:start[k + 1]] % N] = Hv[start[k]:start[k + 1]]
        L = int(plen[k])
        seg = win.pool[win.pre_off[rep[k]]:win.pre_off[rep[k]] + L]
        if pop_pass and cnt0[k] > 64:
            # the popular pass: the prefix walk once per first block (its
            # representative, the first such group here), then each group from
            # the end of the common prefix, k0, with the live set read from the
            # prefix row
            key = int(seg[0])
            if key not in first_block:
                hr = np.sort(h[h >= 1])[::-1]
                P = int(min(L - 1, hr[1] if len(hr) > 1 else 0))
                q = min(L, 1 + 128 * (P // 128 + 1))  # rounds of 128 positions
                cnts = (h[None, :] > np.arange(1, q)[:, None]).sum(1)
                walk += 8 * min(L, 256) + 128 * (q - 1) + int(np.where(cnts > 64, 8 * nw, 2 * cnts).sum())
                walk += 4 * int(cnt0[k])  # the prefix row
                first_block[key] = (seg, q)
            rseg, q = first_block[key]
            lim = min(L, len(rseg), q)
            diff = np.nonzero(seg[:lim] != rseg[:lim])[0]
            k0 = int(diff[0]) if len(diff) else lim
            # staged head, LCP compare, prefix row read, walk from k0, hits, class, record
            hk = np.where(h >= k0, h, 0)
            walk += 8 * min(L, 256) + 16 * k0 + 4 * int(cnt0[k]) + index_walk_bytes(hk, L, nw) \
                + 4 * int(cnt0[k]) + 8 * nw + 4 * int(cnt0[k]) + 8 + 8
            continue
        walk += 8 + index_walk_bytes(h, L, nw) + 4 * int(cnt0[k])
        if cnt0[k] > 64:  # the shared-hit class: bitmap and hits read back, the class word
            walk += 8 * nw + 4 * int(cnt0[k]) + 8
    return claim, walk

def score_bytes(win, r0, hits, grp=None):
    """Algorithmic bytes the scoring pass moves for requests r0 .. r0 +
    len(hits) (the benchmark's policy: D-C-Q, monotone model, no set sizes),
    as (lean scorer's, general scorer's).

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

    grp: per request its group's id ("gid", -1 none), whether the group has a
    record ("has"), a popular row ("pop"), a shared-hit class ("cls", with
    H* "hs" and the group's segment length "gplen"); "grouped"; the group
    hits as sparse pairs ("Hk", "Hv").

    Requests of a popular group with a shared-hit class below their
    segment end take the general kernel's class path: the hand-over entry
    (4 B written by the rows kernel, 4 B read), descriptor, slot, 144 B
    record, result, the 64 largest rooms (1 KB), the holder bitmap, 32 B
    per exception's state and its resume walk, one chunk of 64 key-ordered
    states with their ids, one chunk of thresholds, and the chosen state (a
    lower bound: later chunks and the fallback scan are not counted; the
    chunk summaries and maxima sit in LDS for a wave's whole launch).

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
    if grp is None:
        grp = dict(has=np.zeros(R, bool), pop=np.zeros(R, bool), grouped=np.zeros(R, bool),
                   gid=np.full(R, -1, np.int64), Hk=np.zeros(0, np.int64),
                   Hv=np.zeros(0, np.int64))
    # Holder pairs (hit >= 1), in row order; every per-pair term below is
    # zero on the other pairs.
    pr, pi = np.nonzero(hits)
    ph = hits[pr, pi].astype(np.int64)
    p_elig = room[pi] >= L[pr]

    def per_row(v):
        return np.bincount(pr, weights=v, minlength=R).astype(np.int64)

    room_sorted = np.sort(room)
    nA = N - np.searchsorted(room_sorted, L, side="left")   # eligible instances
    cnt0 = np.bincount(pr, minlength=R)                      # holders of the first block
    ncand = np.bincount(pr, weights=p_elig, minlength=R).astype(np.int64)
    act = nA > 0
    lean = grp["has"] & ~grp["pop"]
    pop = grp["has"] & grp["pop"]
    # popular groups with a shared-hit class, where H* lies below the
    # request's segment end (p0): the class path of the general kernel
    if "cls" in grp:
        p0 = np.minimum(p, grp["gplen"])
        clsp = grp["cls"] & (grp["hs"] < p0)
    else:
        clsp = np.zeros(R, bool)
    pop = pop & ~clsp
    # resume walks of grouped requests: the group's segment hit on the pair
    p_Hg = np.where(grp["gid"][pr] >= 0,
                    _lookup(grp["Hk"], grp["Hv"], np.maximum(grp["gid"][pr], 0) * N + pi), 0)
    p_resume = p_elig & (p_Hg >= p[pr]) & (p[pr] < ell[pr])
    p_rb = np.where(ph > p[pr], PROBE_ROWPOS + 16 * (np.minimum(ph, ell[pr] - 1) - p[pr]) +
                    BUCKET_BYTES * (ph < ell[pr]), PROBE_ROWPOS)
    resume_by = per_row(np.where(p_resume, p_rb, 0))
    # general kernel: per-request parts
    gen = 48 + 512 * levels + np.zeros(R, np.int64)
    gen += np.where(pop, 144 + np.where(act & (ell > 0), 128 + np.where(
        cnt0 <= 64, 10 * cnt0, 8 * nw + 8 * cnt0) + 4 * ncand, 0) + resume_by, 0)
    nogrp = ~grp["has"]
    gen += np.where(nogrp, 8 * np.minimum(ell, 256) + np.where(grp["grouped"], 144, 0), 0)
    gen += np.where(nogrp & act & (ell > 0), 128 + np.where(cnt0 <= 64, 10 * cnt0, 8 * nw + 8 * cnt0), 0)
    few = ncand <= 64
    walk = per_row(np.where(p_elig, PROBE_ROWPOS + 16 * np.minimum(ph, ell[pr] - 1) +
                            BUCKET_BYTES * (ph < ell[pr]), 0))
    gen += np.where(nogrp & act & few & (ell > 1), walk, 0)
    for r in np.nonzero(nogrp & act & ~few & (ell > 1))[0]:
        h_r = hits[r].astype(np.int64)
        gen[r] += index_walk_bytes(np.where(room >= L[r], h_r, 0), int(ell[r]), nw, h_r)
    # lean kernel: per-request parts
    lby = 184 + (0 if small else 32) * cnt0 + resume_by
    lby = np.where(act, lby, 184)
    by = np.where(lean, lby, gen)
    if clsp.any():
        p_exc = (p_Hg >= 1) & (p_Hg != grp["hs"][pr])    # holders off the class hit
        ex_res = per_row(np.where(p_resume & p_exc, p_rb, 0))
        cby = (4 + 4 + 24 + 4 + 8 * 18 + 20 + 64 * 16 + 8 * nw + 32 * per_row(p_exc) + ex_res +
               64 * (4 + 32) + 64 * 16 + 32)
        by = np.where(clsp, cby, by)
    # The recomputation filter: W = max(0, T_pf(n, c) - T_pf(0, L)); a
    # non-holder (n = L) has W = max(0, Z).
    Lf = L.astype(np.float64)
    Z = _tpf(a, Lf, 0.0) - _tpf(a, 0.0, Lf)
    W0 = np.maximum(0.0, Z)
    p_n = (L[pr] - ph * bs).astype(np.float64)
    p_c = (ph * bs).astype(np.float64)
    p_W = np.maximum(0.0, _tpf(a, p_n, p_c) - _tpf(a, 0.0, Lf[pr]))
    n0 = nA - ncand
    Wmin = np.where(n0 > 0, W0, np.inf)
    np.minimum.at(Wmin, pr[p_elig], p_W[p_elig])
    kvc = Z > 0
    with np.errstate(divide="ignore", invalid="ignore"):
        p_rho = (p_W - Wmin[pr]) / Z[pr]
        admit0 = (n0 > 0) & (~kvc | ((W0 - Wmin) / Z <= eta))
    p_inC = p_elig & (~kvc[pr] | (p_rho <= eta))
    by += np.where(lean | clsp, 0, 32 * per_row(p_inC))
    seg = np.searchsorted(ub, A1, side="left")
    seg = np.minimum(seg, len(ub) - 1)
    order0 = np.lexsort((np.arange(N), win.Q, -win.D.astype(np.int64)))
    chunk_lean = 0 if small else 64 * 16

    def dense_rows(rr):
        """Eligibility, holders, new / cached tokens and C membership of the
        candidates of the requests rr, on every instance."""
        h = hits[rr].astype(np.int64)
        el = room[None, :] >= L[rr][:, None]
        hold = h >= 1
        n_ = (L[rr][:, None] - h * bs).astype(np.float64)
        c_ = (h * bs).astype(np.float64)
        W = np.maximum(0.0, _tpf(a, n_, c_) - _tpf(a, 0.0, Lf[rr][:, None]))
        with np.errstate(divide="ignore", invalid="ignore"):
            rho = (W - Wmin[rr][:, None]) / Z[rr][:, None]
        inC_ = el & (~kvc[rr][:, None] | (rho <= eta))
        return el, hold, n_, c_, inC_

    # The zero-hit class per request: which 64-instance chunks of the key
    # order hold a member of T, the first that holds an admitted non-holder,
    # and whether the class is evaluated in full (no member of the class and
    # no candidate in T).
    rows = np.nonzero(act & (admit0 | lean) & ~clsp)[0]
    mono = (beta[:, 2] >= 0).all() and (gam >= 0).all() and a[1] >= 0 and a[3] >= 0

    def tpot0_of(Lt, idx=slice(None)):
        """TPOT of a zero-hit request of Lt tokens on the instances idx."""
        sg = seg[idx]
        t_it = gam[sg] * (beta[sg, 0] + beta[sg, 1] * A1[idx] + beta[sg, 2] * (win.S[idx] + Lt))
        return t_it, t_it + np.where(A1[idx] > 1, _tpf(a, Lt, 0.0) / lout1, 0.0)

    def dense(rr):
        """Every instance of every request of rr (any model)."""
        k = len(rr)
        el, hold, _, _, _ = dense_rows(rr)
        t_iter, tpot0 = tpot0_of(L[rr].astype(np.float64)[:, None])
        below = tpot0 < tau
        zero = el & ~hold
        feas = np.zeros((k, n1 * 64), bool)
        feas[:, :N] = (el & below)[:, order0]
        passing = feas.reshape(k, n1, 64).any(2)
        okm = (zero & below)[:, order0]
        found = okm.any(1)
        cs = np.where(found, np.argmax(okm, 1) // 64, n1 - 1)
        return found, cs, passing

    def finish(rr, found, cs, passing):
        k = len(rr)
        npass = np.cumsum(passing, 1)[np.arange(k), cs]
        lean_r, adm = lean[rr], admit0[rr]
        spec = lean_r & ~adm          # only the speculative first chunk
        add = np.zeros(k, np.int64)
        add[spec] = np.where(passing[spec].any(1), chunk_lean, 0)
        m = lean_r & adm
        add[m] = chunk_lean * npass[m] + (0 if small else 32 * found[m])
        m = ~lean_r
        add[m] = 256 * (cs[m] // 64 + 1) + 1024 * npass[m]
        # No member of the class is in T: it is evaluated in full only when
        # no candidate is in T either.
        need = ~found & ~spec
        if need.any():
            rn = rr[need]
            el, hold, n_, c_, inC_ = dense_rows(rn)
            t_iter = tpot0_of(L[rn].astype(np.float64)[:, None])[0]
            tp = t_iter + np.where(A1[None, :] > 1, _tpf(a, n_, c_) / lout1, 0.0)
            none_t = ~(el & hold & inC_ & (tp < tau)).any(1)
            full = np.zeros(k, bool)
            full[need] = none_t
            nz = np.zeros(k, np.int64)
            nz[need] = (el & ~hold).sum(1)
            add += np.where(full & lean_r, 0 if small else 32 * N + 32, 0)
            add += np.where(full & ~lean_r, 8 * N + 32 * nz, 0)
        by[rr] += add

    if mono and len(rows):
        # Monotone model: "eligible and TPOT below tau" for a zero-hit request
        # of L tokens is L <= thr_i = min(room_i, the longest admitted L), so
        # the first admitted instance in key order comes from a prefix
        # maximum; rows whose first admitted instance holds the first block
        # take the dense path.
        ell_hi = int(max(1, (win.pre_len.astype(np.int64) + win.tail_len).max()))
        lo = np.full(N, -1, np.int64)           # admitted at lo blocks (-1: none)
        hi = np.full(N, ell_hi + 1, np.int64)   # refused at hi blocks
        ok_hi = tpot0_of(float(ell_hi * bs))[1] < tau
        lo[ok_hi] = ell_hi
        while (hi > lo + 1).any():
            open_ = hi > lo + 1
            mid = np.where(open_, (lo + hi) // 2, lo)
            okm = tpot0_of((np.maximum(mid, 0) * bs).astype(np.float64))[1] < tau
            lo = np.where(open_ & okm, mid, lo)
            hi = np.where(open_ & ~okm, mid, hi)
        lmax = np.where(lo >= 0, lo * bs, -1)
        thr = np.minimum(room, lmax)
        thr_o = np.full(n1 * 64, -2, np.int64)
        thr_o[:N] = thr[order0]
        cmax = thr_o.reshape(n1, 64).max(1)
        pmax = np.maximum.accumulate(thr_o)
        p0 = np.searchsorted(pmax, L[rows], side="left")   # first position admitting L
        anyadm = p0 < N
        first = order0[np.minimum(p0, N - 1)]
        holder_first = anyadm & (hits[rows, first] >= 1)
        rf = rows[~holder_first]
        found = anyadm[~holder_first]
        cs = np.where(found, p0[~holder_first] // 64, n1 - 1)
        finish(rf, found, cs, cmax[None, :] >= L[rf][:, None])
        rows = rows[holder_first]
    for b0 in range(0, len(rows), 512):
        rr = rows[b0:b0 + 512]
        found, cs, passing = dense(rr)
        finish(rr, found, cs, passing)
    return int(by[lean].sum()), int(by[~lean].sum())


def survey_pair_bytes(win, r0, pr, pi, ph, n_rows, N):
    """The per-window algorithmic bytes of a walk of every capacity-eligible
    (request, instance) pair, for requests r0 .. r0 + n_rows: 64 B per probe,
    min(hit + 1, chain length) probes per eligible pair, plus 8 B per
    request-chain block read (min(longest eligible hit + 1, chain length)),
    plus 20 B of result per request.  (The instances' 24 B of state are
    added once per window by the caller.)"""
    import numpy as np
    pol = win.policy
    bs, bmax, kv = int(pol["block_tokens"]), int(pol["b_max"]), int(pol["kv_cap_tokens"])
    A1 = win.D.astype(np.int64) + win.Q + 1
    room = np.where(A1 <= bmax, kv - win.S, -1)
    ell = (win.pre_len.astype(np.int64) + win.tail_len)[r0:r0 + n_rows]
    L = ell * bs
    nA = N - np.searchsorted(np.sort(room), L, side="left")
    el = room[pi] >= L[pr]
    ncand = np.bincount(pr, weights=el, minlength=n_rows).astype(np.int64)
    probes = (nA - ncand) * (ell > 0) + np.bincount(
        pr, weights=np.where(el, np.minimum(ph + 1, ell[pr]), 0), minlength=n_rows).astype(np.int64)
    hmax = np.zeros(n_rows, np.int64)
    np.maximum.at(hmax, pr[el], ph[el])
    chain = np.where(nA > 0, np.minimum(hmax + 1, ell), 0)
    return int(64 * probes.sum() + 8 * chain.sum() + 20 * n_rows)


def algorithmic_bytes(sc, win, d_pool, chunk_pairs=1 << 25):
    """Algorithmic bytes of every kernel of one scoring call (claim pass,
    group walk, lean scorer, general scorer), of the exhaustive probe
    kernel over the window, and the per-pair figure, from the exhaustive
    per-pair hits exported chunk by chunk (untimed)."""
    import numpy as np
    import torch
    import paper_2609_33224_amd as ps
    N = win.n_inst
    gid, rep, plen = group_info(win)
    Hk, Hv = group_segment_hits(sc, win, d_pool, rep, plen)
    G = len(rep)
    cnt = np.bincount(Hk // N, minlength=G) if G else np.zeros(0, np.int64)
    # every group gets a result: a record, or a popular row (the area holds
    # 64 MiB / (4 n_inst) rows, more than any benchmark window needs)
    g_pop = cnt > GROUP_HOLD
    assert int(g_pop.sum()) <= (64 << 20) // (4 * N)
    claim_b, walk_b = group_pass_bytes(win, gid, rep, plen, Hk, Hv)
    g_cls, g_hs = group_classes(Hk, Hv, G, N)
    chunk = max(1, min(win.n_req, chunk_pairs // N))
    reqs = ps.pack_reqs(win.pre_off, win.pre_len, win.tail_off, win.tail_len)
    d_hits = torch.empty(chunk * N, dtype=torch.int32, device="cuda")
    lean_b = gen_b = probe_b = n_probes = pair_b = 0
    for r0 in range(0, win.n_req, chunk):
        n = min(chunk, win.n_req - r0)
        d_r = ps.to_device_bytes(reqs[r0:r0 + n])
        sc.hits_dev(d_pool, len(win.pool), d_r, n, d_hits)
        torch.cuda.synchronize()
        hits = d_hits[: n * N].cpu().numpy().view(np.uint32).reshape(n, N)
        pr, pi = np.nonzero(hits)
        ph = hits[pr, pi].astype(np.int64)
        b, p_ = probe_bytes(win, r0, pr, ph, n, N)
        probe_b += b
        n_probes += p_
        pair_b += survey_pair_bytes(win, r0, pr, pi, ph, n, N)
        gc = gid[r0:r0 + n]
        grouped = gc >= 0
        gi = np.maximum(gc, 0)
        if G:
            pop = grouped & g_pop[gi]
            grp = dict(has=grouped, pop=pop, grouped=grouped, gid=gc, Hk=Hk, Hv=Hv,
                       cls=pop & g_cls[gi], hs=g_hs[gi], gplen=plen[gi])
        else:
            grp = None
        lb, gb = score_bytes(win, r0, hits, grp)
        lean_b += lb
        gen_b += gb
    pair_b += 24 * N
    # the key-only variant: 8 bytes (the key) per probe instead of the bucket
    probe_key = probe_b - n_probes * (BUCKET_BYTES - 8)
    return dict(claim=claim_b, walk=walk_b, lean=lean_b, general=gen_b, probe=probe_b,
                probe_key_only=probe_key, probes=n_probes, pairs=pair_b, groups=G,
                popular_groups=int(g_pop.sum()))


def traffic_for(workload: str, src_hash: str):
    """The committed counter summary for this workload, if it was taken on
    these kernel sources."""
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
    """The oracle on the host cores over a leading slice of the window sized
    from a short timed slice to fill about `budget_s` seconds (the whole
    window, repeated, when it takes less)."""
    import oracle
    o = oracle.Oracle.from_window(win)
    threads = oracle.max_threads()
    n0 = min(win.n_req, 2048)
    t0 = time.perf_counter()
    o.window_score(win.subset(range(n0)), nthreads=threads)
    per_req = (time.perf_counter() - t0) / n0
    if per_req * win.n_req < budget_s:
        reps = max(1, int(budget_s / max(per_req * win.n_req, 1e-3)))
        t0 = time.perf_counter()
        for _ in range(reps):
            o.window_score(win, nthreads=threads)
        dt = (time.perf_counter() - t0) / reps
        n, sample = win.n_req, (f"whole window ({win.n_req} requests x {win.n_inst} instances), "
                                f"{reps} repetitions")
    else:
        n = max(n0, min(win.n_req, int(budget_s / per_req)))
        sub = win.subset(range(n))
        t0 = time.perf_counter()
        o.window_score(sub, nthreads=threads)
        dt = time.perf_counter() - t0
        sample = (f"first {n} of {win.n_req} requests x {win.n_inst} instances, once "
                  f"(sized from a timed slice of {n0})")
    # one core, on a leading slice of about two seconds
    n1 = max(1, min(win.n_req, int(2.0 / max(per_req * threads, 1e-9))))
    t0 = time.perf_counter()
    o.window_score(win.subset(range(n1)), nthreads=1)
    dt1 = time.perf_counter() - t0
    o.close()
    return dict(value=n * win.n_inst / dt, unit="candidate evals/s", cores=threads,
                kind="oracle", decisions_per_s=n / dt, seconds=dt, sample=sample,
                one_core=dict(value=n1 * win.n_inst / dt1, unit="candidate evals/s", cores=1,
                              decisions_per_s=n1 / dt1,
                              sample=f"first {n1} of {win.n_req} requests x {win.n_inst} "
                                     f"instances, once"))


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
    o.close()
    o = oracle.Oracle.from_window(win)
    t0 = time.perf_counter()
    o.window_schedule(win.subset(range(n)) if n < win.n_req else win)
    dt = time.perf_counter() - t0
    o.close()
    return dict(value=n / dt, unit="decisions/s", cores=1, kind="oracle",
                sample=(f"first {n} of {win.n_req} requests, per arrival, once" if n < win.n_req
                        else f"whole window ({win.n_req} requests), per arrival, once"))


def sequential_block(sc, win, model, d_pool, d_reqs, n, snap, reps, stream):
    """Algorithm 1 per arrival (ps_schedule_window_dev) on the window's first
    n requests from the loaded state, and the herding of the snapshot
    placements of the same requests: those placements replayed in arrival
    order (ps_replay_window_dev)."""
    import numpy as np
    import torch
    import paper_2609_33224_amd as ps

    def reload():
        sc.load(win.n_inst, win.cap, win.blk_off, win.blk, win.D, win.Q, win.P, win.S, model)
        torch.cuda.synchronize()

    snap_all = snap[:n]
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
    n_spec, n_full = sc.schedule_stats()
    # the same leading requests with every request scored in full by the
    # one scheduler workgroup (no speculative batches), for comparison
    n_off = min(n, 4096)
    sc.set_schedule_speculation(0)
    reload()
    t0 = time.perf_counter()
    sc.schedule_dev(d_pool, len(win.pool), d_reqs, n_off, d_out, None, stream)
    off_s = time.perf_counter() - t0
    sc.set_schedule_speculation(256)
    # The replay stops before the first placement that would take an
    # instance's queue past its 12-bit limit (snapshot herding can).
    n_rep, q = n, win.Q.astype(np.int64).copy()
    for k, i in enumerate(snap_all["instance"]):
        if i >= 0:
            q[i] += 1
            if q[i] > 4095:
                n_rep = k
                break
    reload()
    d_inst = torch.from_numpy(np.ascontiguousarray(snap_all["instance"][:n_rep], np.int32)).to("cuda")
    t0 = time.perf_counter()
    if n_rep:
        sc.replay_dev(d_pool, len(win.pool), d_reqs, n_rep, d_inst, d_out, stream)
    replay_s = time.perf_counter() - t0
    rep = ps.results_from_device(d_out)[:n_rep]
    snap_r = snap_all[:n_rep]
    tau = float(np.float32(win.policy["tpot_slo"]))
    fb = ps.PS_R_FALLBACK
    ok_snap = (snap_r["instance"] >= 0) & ((snap_r["flags"] & fb) == 0)
    ok_seq = (seq["instance"] >= 0) & ((seq["flags"] & fb) == 0)
    per_snap = np.bincount(snap_all["instance"][snap_all["instance"] >= 0], minlength=win.n_inst)
    per_seq = np.bincount(seq["instance"][seq["instance"] >= 0], minlength=win.n_inst)
    ms = float(np.mean(times)) * 1e3
    return {
        "entry": "ps_schedule_window_dev: Algorithm 1 per arrival (batches of 256: hits pass, "
                 "every request scored in parallel against the batch's starting state, then "
                 "one workgroup checks each result against the instances placed on since, "
                 "decides and commits in arrival order; rebuild of the derived data)",
        "requests": n, "of_window": win.n_req,
        "ms_per_call": ms, "decisions_per_s": n / (ms * 1e-3),
        "us_per_decision": ms * 1e3 / n, "reps": reps,
        "decided_from_speculation": n_spec, "scored_in_full": n_full,
        "without_speculation": {"requests": n_off, "ms_per_call": off_s * 1e3,
                                "us_per_decision": off_s * 1e6 / max(n_off, 1)},
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


KERNELS = ("group_claim_kernel", "group_kernel", "lean_rows_kernel", "score_kernel")
KERNEL_ROLE = {
    "group_claim_kernel": "prefix-group claim pass (each request's group slot, leader lists)",
    "group_kernel": "prefix-group walk (each shared segment walked once on every holder of its "
                    "first block; groups whose first block has a holder bitmap in the popular "
                    "pass beside it, the walk then on a second stream; timed from the claim "
                    "pass's end to the join of both on the calling stream)",
    "lean_rows_kernel": "scorer, four requests per wave (hits from the group records, latency "
                        "model, filters, packing key, argmin)",
    "score_kernel": "general scorer (requests the lean scorer left: popular groups)",
}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c5", choices=sorted(WORKLOAD_NAMES))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the CPU baseline (sized from a timed slice)")
    ap.add_argument("--sequential-requests", type=int, default=16384,
                    help="leading requests of the window scheduled per arrival (0: skip)")
    ap.add_argument("--sequential-reps", type=int, default=2)
    ap.add_argument("--skip-bytes", action="store_true",
                    help="skip the algorithmic byte counts (roofline fields null; for counter runs)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run 5 device-to-device copies of this many MiB (a plain copy "
                         "kernel of known size, to scale the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the scorer runs on one GPU; --gpus {args.gpus} is not supported "
              "(more GPUs would each score a slice of the requests against replicated "
              "instance tables)", file=sys.stderr)
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

    def say(msg):
        print(f"bench: {msg}", file=sys.stderr, flush=True)

    say(f"generating {args.workload}")
    win = synth.generate(args.workload, seed=args.seed)
    sc = ps.Scorer(0)
    m = ps.make_model(win.alpha, win.seg_ub, win.beta, win.gamma, win.policy["eta"],
                      win.policy["tpot_slo"], win.policy["ttft_floor"], win.policy["lout"],
                      win.policy["block_tokens"], win.policy["b_max"],
                      win.policy["kv_cap_tokens"], win.policy["flags"], win.policy["rand_seed"])
    say("loading the instances")
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
        nb = None
    else:
        say("counting algorithmic bytes")
        nb = algorithmic_bytes(sc, win, d_pool)
    t0 = time.perf_counter()
    sc.score(win.pool, reqs)
    host_call_s = time.perf_counter() - t0

    # the exhaustive per-instance probe kernel (ps_probe_hits_dev), timed alone
    say("timing the exhaustive probe kernel")
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
    say(f"timing {args.steps} steps")
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
    step_ev = [a.elapsed_time(b) for a, b in ev]
    step_avg = float(np.mean(step_ev))
    # The same steps again with the library's events around each of its
    # launches, recorded on the launch stream.
    sc.set_timing(True)
    for _ in range(args.steps):
        sc.score_dev(d_pool, len(win.pool), d_reqs, win.n_req, d_out, None, stream)
    n_timed, kern_ms = sc.read_kernel_timing()
    sc.set_timing(False)

    evals = win.n_req * win.n_inst
    src_hash = kernel_source_hash()
    from paper_2609_33224_amd import build as ps_build
    lib_id = ps.ps_build_id()
    lib_fresh = lib_id == ps_build.source_hash()
    if not lib_fresh:
        say(f"libpackserve.so was built from other sources ({lib_id}); rebuild it "
            "(__graft_entry__.build()); counter bytes are not applied")
    tent = (traffic_for(args.workload, src_hash) or {}) if lib_fresh else {}
    tk = tent.get("kernels", {})

    def rate(nbytes, ms):
        return nbytes / (ms * 1e-3) / 1e9 if nbytes is not None and ms and ms > 0 else None

    kb = dict(zip(KERNELS, (nb["claim"], nb["walk"], nb["lean"], nb["general"]) if nb else (None,) * 4))
    kernels = {}
    for name, ms in zip(KERNELS, kern_ms):
        ach = rate(kb[name], ms)
        kernels[name] = {"role": KERNEL_ROLE[name], "ms_avg": ms, "algorithmic_bytes": kb[name],
                         "achieved_GBs": ach,
                         "frac_of_hbm_peak": ach / HBM_PEAK_GBS if ach is not None else None,
                         "counter_bytes": (tk.get(name) or {}).get("bytes_per_launch")}
    dom = max(KERNELS, key=lambda k: kernels[k]["ms_avg"])
    dk = kernels[dom]
    call_bytes = sum(kb.values()) if nb else None
    call_gbs = rate(call_bytes, ms_per_step)
    probe_gbs = rate(nb["probe"] if nb else None, probe_ms)
    probe_meas = tent.get("probe_bytes_per_window")
    pair_gbs = rate(nb["pairs"] if nb else None, ms_per_step)
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
        "step_ms_events_median": float(np.median(step_ev)),
        "roofline": {"bound": "hbm", "achieved": dk["achieved_GBs"], "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": dk["frac_of_hbm_peak"], "traffic": dk["counter_bytes"],
                     "kernel": dom},
        "kernels": kernels,
        "kernel_timed_calls": n_timed,
        "call": {"algorithmic_bytes": call_bytes, "achieved_GBs": call_gbs,
                 "frac_of_hbm_peak": call_gbs / HBM_PEAK_GBS if call_gbs is not None else None},
        "per_pair_walk": {
            "about": "bytes of walking every capacity-eligible request x instance pair with 64 B "
                     "bucket probes (the scoring call does not: the prefix index and the group "
                     "pass skip them), over the step's time",
            "bytes": nb["pairs"] if nb else None, "GBs_over_step": pair_gbs,
            "frac_of_hbm_peak": pair_gbs / HBM_PEAK_GBS if pair_gbs is not None else None},
        "groups": {"groups": nb["groups"] if nb else None,
                   "popular_groups": nb["popular_groups"] if nb else None},
        "probe_kernel": {"kernel": "ps_probe_hits_dev (every request x instance probed)",
                         "ms_per_window": probe_ms, "probes": nb["probes"] if nb else None,
                         "algorithmic_bytes": nb["probe"] if nb else None,
                         "achieved_GBs": probe_gbs,
                         "algorithmic_bytes_key_only": nb["probe_key_only"] if nb else None,
                         "achieved_GBs_key_only": rate(nb["probe_key_only"] if nb else None, probe_ms),
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
    n_seq = min(args.sequential_requests, win.n_req)
    if n_seq > 0:
        say(f"per-arrival scheduling of the first {n_seq} requests")
        out["sequential"] = sequential_block(sc, win, m, d_pool, d_reqs, n_seq, res,
                                             args.sequential_reps, stream)
    sc.close()
    if not args.no_cpu_baseline:
        say("timing the CPU oracle")
        out["cpu_baseline"] = cpu_baseline(win, args.cpu_budget)
        if n_seq > 0:
            out["cpu_baseline"]["sequential"] = cpu_sequential_baseline(
                win.subset(range(n_seq)), args.cpu_budget / 3)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
