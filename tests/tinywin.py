"""Hand-built tiny windows for pins and edge cases (data marshalling only).

A tiny window is a ``synth.Window`` assembled from explicit per-instance
block lists and explicit request chains, so that tests can state exactly
which blocks each instance holds.
"""
import numpy as np

from synth import Window

DEFAULT_POLICY = dict(eta=0.5, tpot_slo=0.030, ttft_floor=2.0, lout=556.0, block_tokens=16,
                      b_max=64, kv_cap_tokens=1_000_000, flags=0, rand_seed=0)


def make_window(sets, chains, D, Q, P, S, alpha, seg_ub, beta, gamma, cap=None, **policy):
    """sets: list (per instance) of lists of uint64 block hashes.
    chains: list (per request) of lists of block hashes, or of
    (prefix, tail) pairs to use the two-segment descriptor."""
    n_inst = len(sets)
    lens = [len(s) for s in sets]
    blk_off = np.zeros(n_inst + 1, np.int64)
    blk_off[1:] = np.cumsum(lens)
    blk = np.array([h for s in sets for h in s], dtype=np.uint64)
    pool, pre_off, pre_len, tail_off, tail_len = [], [], [], [], []
    for ch in chains:
        if isinstance(ch, tuple):
            pre, tail = ch
        else:
            pre, tail = ch, []
        pre_off.append(len(pool))
        pre_len.append(len(pre))
        pool.extend(pre)
        tail_off.append(len(pool))
        tail_len.append(len(tail))
        pool.extend(tail)
    pol = dict(DEFAULT_POLICY)
    pol.update(policy)
    return Window(
        n_inst=n_inst, cap=int(cap if cap is not None else max(max(lens, default=0), 1)),
        blk_off=blk_off, blk=blk,
        D=np.asarray(D, np.int32), Q=np.asarray(Q, np.int32),
        P=np.asarray(P, np.int64), S=np.asarray(S, np.int64),
        alpha=np.asarray(alpha, np.float64), seg_ub=np.asarray(seg_ub, np.int32),
        beta=np.asarray(beta, np.float64).reshape(-1, 3), gamma=np.asarray(gamma, np.float64),
        policy=pol,
        pool=np.array(pool, dtype=np.uint64),
        pre_off=np.array(pre_off, np.int64), pre_len=np.array(pre_len, np.int32),
        tail_off=np.array(tail_off, np.int64), tail_len=np.array(tail_len, np.int32),
        meta={},
    )


def chain_hashes(n, base=1000):
    """n distinct nonzero block hashes."""
    return [base + 7 * j + 1 for j in range(n)]


def make_window_pool(sets, pool, reqs, D, Q, P, S, alpha, seg_ub, beta, gamma, cap=None,
                     **policy):
    """Like make_window, with an explicit hash pool and descriptors
    (pre_off, pre_len, tail_off, tail_len), so that several requests can
    share one pool segment."""
    w = make_window(sets, [], D, Q, P, S, alpha, seg_ub, beta, gamma, cap=cap, **policy)
    w.pool = np.asarray(pool, dtype=np.uint64)
    d = np.asarray(reqs, dtype=np.int64).reshape(-1, 4)
    w.pre_off, w.pre_len = d[:, 0].copy(), d[:, 1].astype(np.int32)
    w.tail_off, w.tail_len = d[:, 2].copy(), d[:, 3].astype(np.int32)
    return w
