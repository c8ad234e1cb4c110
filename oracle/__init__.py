"""CPU oracle for the PackServe window scorer -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package.  The GPU library and its Python binding never
import it, and the two share no code.  The arithmetic lives in
``oracle.cpp`` (plain C++, fp64, OpenMP over requests); this module only
builds it and marshals numpy arrays.

See the header of ``oracle.cpp`` for what each function follows in the
paper, what pins it, and which readings are "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
# A test that plants a mistake in a copy of the oracle points this at the
# mutant build; nothing else sets it.
if os.environ.get("PS_ORACLE_MUTANT_LIB"):
    _LIB_PATH = os.environ["PS_ORACLE_MUTANT_LIB"]
_lib = None

F_TTFT_ADMIT, F_NO_KVC_FILTER, F_NO_TPOT_FILTER, F_FALLBACK_DCQ = 1, 2, 4, 8
SEL_DCQ, SEL_D, SEL_DQ, SEL_DC, SEL_DQC, SEL_HCQ, SEL_RANDOM, SEL_LMETRIC = range(8)


def selector_flags(sel: int) -> int:
    return (int(sel) & 0xF) << 8
R_REJECT, R_FALLBACK, R_TTFT_MISS = 1, 2, 4
# Near-boundary bits (see oracle.cpp): the decision, the TTFT_MISS flag, or
# only |C| / |T| may be decided by rounding.
NB_RHO, NB_TPOT, NB_TTFT, NB_Z, NB_MISSFLAG, NB_HEADROOM, NB_SIZES = 1, 2, 4, 8, 16, 32, 64
NB_DECISION = NB_RHO | NB_TPOT | NB_TTFT | NB_Z | NB_HEADROOM
NB_SET_C = NB_RHO | NB_Z            # |C| (and so |T|) may be decided by rounding
NB_UNSURE_SHIFT = 16                # nb >> 16: candidates whose T membership is unsure


def build(verbose: bool = False) -> str:
    """Compile ``oracle.cpp`` into ``liboracle.so`` (always recompiles)."""
    src = os.path.join(_HERE, "oracle.cpp")
    tmp = _LIB_PATH + ".tmp"
    cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-shared", "-fPIC", "-o", tmp, src]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    global _lib
    _lib = None
    return _LIB_PATH


class Model(ctypes.Structure):
    """fp64 model/policy; field meanings as in ``oracle.cpp``."""
    _fields_ = [
        ("alpha", ctypes.c_double * 6),
        ("n_seg", ctypes.c_int32),
        ("seg_ub", ctypes.c_int32 * 32),
        ("beta", (ctypes.c_double * 3) * 32),
        ("gamma", ctypes.c_double * 32),
        ("eta", ctypes.c_double), ("tau", ctypes.c_double),
        ("ttft_floor", ctypes.c_double), ("lout", ctypes.c_double),
        ("block_tokens", ctypes.c_int32), ("b_max", ctypes.c_int32),
        ("kv_cap", ctypes.c_int64),
        ("flags", ctypes.c_uint32),
        ("rand_seed", ctypes.c_uint64),
    ]


def make_model(alpha, seg_ub, beta, gamma, eta, tau, ttft_floor, lout, block_tokens, b_max,
               kv_cap, flags=0, rand_seed=0) -> Model:
    """Fill an oracle model.  Values are taken as given (Python floats are
    fp64; pass fp32 arrays to reproduce the interface precision exactly)."""
    m = Model()
    for k in range(6):
        m.alpha[k] = float(alpha[k])
    m.n_seg = len(seg_ub)
    for s in range(len(seg_ub)):
        m.seg_ub[s] = int(seg_ub[s])
        for k in range(3):
            m.beta[s][k] = float(beta[s][k])
        m.gamma[s] = float(gamma[s])
    m.eta, m.tau, m.ttft_floor, m.lout = float(eta), float(tau), float(ttft_floor), float(lout)
    m.block_tokens, m.b_max, m.kv_cap, m.flags = int(block_tokens), int(b_max), int(kv_cap), int(flags)
    m.rand_seed = int(rand_seed) & 0xFFFFFFFFFFFFFFFF
    return m


def model_of(win, **policy_overrides) -> Model:
    """The oracle model of a generated window (fp32 coefficients widened)."""
    pol = dict(win.policy)
    pol.update(policy_overrides)
    return make_model(win.alpha.astype(np.float64), win.seg_ub, win.beta.astype(np.float64),
                      win.gamma.astype(np.float64), np.float32(pol["eta"]),
                      np.float32(pol["tpot_slo"]), np.float32(pol["ttft_floor"]),
                      np.float32(pol["lout"]), pol["block_tokens"], pol["b_max"],
                      pol["kv_cap_tokens"], pol.get("flags", 0), pol.get("rand_seed", 0))


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is missing: run oracle.build() first")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.orc_load.argtypes = [i32, i32, vp, vp, vp, vp, vp, vp, ctypes.POINTER(vp)]
    lib.orc_load.restype = ctypes.c_int
    lib.orc_free.argtypes = [vp]
    lib.orc_free.restype = None
    lib.orc_hits.argtypes = [vp, vp, vp, vp, vp, vp, i32, vp, i32]
    lib.orc_hits.restype = ctypes.c_int
    lib.orc_score.argtypes = [vp, ctypes.POINTER(Model), vp, vp, vp, vp, vp, i32,
                              vp, vp, vp, vp, vp, vp, vp, i32]
    lib.orc_score.restype = ctypes.c_int
    lib.orc_commit.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, i32, ctypes.POINTER(i64)]
    lib.orc_commit.restype = ctypes.c_int
    lib.orc_schedule.argtypes = [vp, ctypes.POINTER(Model), vp, vp, vp, vp, vp, i32,
                                 vp, vp, vp, vp, vp, vp, vp, vp, ctypes.POINTER(i64)]
    lib.orc_schedule.restype = ctypes.c_int
    lib.orc_replay.argtypes = [vp, ctypes.POINTER(Model), vp, vp, vp, vp, vp, vp, i32,
                               vp, vp, vp, ctypes.POINTER(i64)]
    lib.orc_replay.restype = ctypes.c_int
    lib.orc_state.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.orc_state.restype = ctypes.c_int
    lib.orc_explain.argtypes = [vp, ctypes.POINTER(Model), vp, i32] + [vp] * 8
    lib.orc_explain.restype = ctypes.c_int
    lib.orc_feedback_decode.argtypes = [ctypes.POINTER(Model), vp, vp, vp, i32]
    lib.orc_feedback_decode.restype = ctypes.c_int
    lib.orc_feedback_output.argtypes = [vp, ctypes.POINTER(Model), vp, i32, i32]
    lib.orc_feedback_output.restype = ctypes.c_int
    lib.orc_apply_events.argtypes = [vp, vp, vp, vp, i32]
    lib.orc_apply_events.restype = ctypes.c_int
    lib.orc_max_threads.argtypes = []
    lib.orc_max_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


@dataclass
class Decisions:
    inst: np.ndarray   # int32, -1 = reject
    hit: np.ndarray    # int32 blocks
    ttft: np.ndarray   # float64 s
    tpot: np.ndarray   # float64 s
    flags: np.ndarray  # uint32 R_* bits
    sizes: np.ndarray  # uint32 [n_req, 3] = |A|, |C|, |T|
    nb: np.ndarray     # uint32 NB_* bits


class Oracle:
    """A snapshot of the instance pool held by the oracle."""

    def __init__(self, n_inst, cap, blk_off, blk, D, Q, P, S):
        lib = _load()
        self._keep = [_c(blk_off, np.int64), _c(blk, np.uint64), _c(D, np.int32),
                      _c(Q, np.int32), _c(P, np.int64), _c(S, np.int64)]
        h = ctypes.c_void_p()
        rc = lib.orc_load(int(n_inst), int(cap), *[k[1] for k in self._keep], ctypes.byref(h))
        self._keep = None
        if rc != 0:
            raise MemoryError("oracle snapshot allocation failed")
        self._h = h
        self.n_inst = int(n_inst)

    @classmethod
    def from_window(cls, win) -> "Oracle":
        return cls(win.n_inst, win.cap, win.blk_off, win.blk, win.D, win.Q, win.P, win.S)

    def close(self):
        if getattr(self, "_h", None):
            _load().orc_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _reqs(self, pool, pre_off, pre_len, tail_off, tail_len):
        arrs = [_c(pool, np.uint64), _c(pre_off, np.int64), _c(pre_len, np.int32),
                _c(tail_off, np.int64), _c(tail_len, np.int32)]
        return arrs, [a[1] for a in arrs]

    def hits(self, pool, pre_off, pre_len, tail_off, tail_len, nthreads=0) -> np.ndarray:
        keep, ptrs = self._reqs(pool, pre_off, pre_len, tail_off, tail_len)
        n = len(keep[1][0])
        out = np.zeros((n, self.n_inst), dtype=np.uint32)
        _load().orc_hits(self._h, *ptrs, n, out.ctypes.data, int(nthreads))
        return out

    def score(self, model: Model, pool, pre_off, pre_len, tail_off, tail_len,
              nthreads=0) -> Decisions:
        keep, ptrs = self._reqs(pool, pre_off, pre_len, tail_off, tail_len)
        n = len(keep[1][0])
        d = Decisions(inst=np.zeros(n, np.int32), hit=np.zeros(n, np.int32),
                      ttft=np.zeros(n, np.float64), tpot=np.zeros(n, np.float64),
                      flags=np.zeros(n, np.uint32), sizes=np.zeros((n, 3), np.uint32),
                      nb=np.zeros(n, np.uint32))
        _load().orc_score(self._h, ctypes.byref(model), *ptrs, n, d.inst.ctypes.data,
                          d.hit.ctypes.data, d.ttft.ctypes.data, d.tpot.ctypes.data,
                          d.flags.ctypes.data, d.sizes.ctypes.data, d.nb.ctypes.data,
                          int(nthreads))
        return d

    def schedule(self, model: Model, pool, pre_off, pre_len, tail_off, tail_len, follow=None):
        """Algorithm 1 per arrival (the snapshot moves to the final state).
        ``follow``: another implementation's placements, committed instead of
        the oracle's own where its decision is near a boundary and they differ
        (they must be capacity-eligible).  Returns (Decisions, dropped)."""
        keep, ptrs = self._reqs(pool, pre_off, pre_len, tail_off, tail_len)
        n = len(keep[1][0])
        fp = None
        if follow is not None:
            fa, fp = _c(follow, np.int32)
            assert len(fa) == n
            keep.append((fa, fp))
        d = Decisions(inst=np.zeros(n, np.int32), hit=np.zeros(n, np.int32),
                      ttft=np.zeros(n, np.float64), tpot=np.zeros(n, np.float64),
                      flags=np.zeros(n, np.uint32), sizes=np.zeros((n, 3), np.uint32),
                      nb=np.zeros(n, np.uint32))
        dropped = ctypes.c_int64()
        rc = _load().orc_schedule(self._h, ctypes.byref(model), *ptrs, n, d.inst.ctypes.data,
                                  d.hit.ctypes.data, d.ttft.ctypes.data, d.tpot.ctypes.data,
                                  d.flags.ctypes.data, d.sizes.ctypes.data, d.nb.ctypes.data,
                                  fp, ctypes.byref(dropped))
        if rc != 0:
            raise ValueError("a followed placement is not capacity-eligible")
        return d, int(dropped.value)

    def replay(self, model: Model, pool, pre_off, pre_len, tail_off, tail_len, inst):
        """Latencies of given placements at their arrival, committing each.
        Returns (hit, ttft, tpot, dropped)."""
        keep, ptrs = self._reqs(pool, pre_off, pre_len, tail_off, tail_len)
        ia, ip = _c(inst, np.int32)
        n = len(ia)
        hit = np.zeros(n, np.int32)
        ttft, tpot = np.zeros(n), np.zeros(n)
        dropped = ctypes.c_int64()
        _load().orc_replay(self._h, ctypes.byref(model), *ptrs, ip, n, hit.ctypes.data,
                           ttft.ctypes.data, tpot.ctypes.data, ctypes.byref(dropped))
        return hit, ttft, tpot, int(dropped.value)

    def commit(self, pool, pre_off, pre_len, tail_off, tail_len, inst, block_tokens=16) -> int:
        keep, ptrs = self._reqs(pool, pre_off, pre_len, tail_off, tail_len)
        ia, ip = _c(inst, np.int32)
        dropped = ctypes.c_int64()
        _load().orc_commit(self._h, *ptrs, ip, len(ia), int(block_tokens), ctypes.byref(dropped))
        return int(dropped.value)

    def state(self):
        n = self.n_inst
        D, Q = np.zeros(n, np.int32), np.zeros(n, np.int32)
        P, S, sz = np.zeros(n, np.int64), np.zeros(n, np.int64), np.zeros(n, np.int64)
        _load().orc_state(self._h, D.ctypes.data, Q.ctypes.data, P.ctypes.data, S.ctypes.data,
                          sz.ctypes.data)
        return dict(D=D, Q=Q, P=P, S=S, set_size=sz)

    def apply_events(self, inst, kind, tokens) -> int:
        """Response-path transitions; returns 0, -1 (bad event) or -5 (range)."""
        i_, ip = _c(inst, np.int32)
        k_, kp = _c(kind, np.int32)
        t_, tp = _c(tokens, np.int64)
        return int(_load().orc_apply_events(self._h, ip, kp, tp, len(i_)))

    def feedback_output(self, model: Model, out_len, window=1024) -> None:
        o_, op = _c(out_len, np.int32)
        _load().orc_feedback_output(self._h, ctypes.byref(model), op, len(o_), int(window))

    def explain(self, model: Model, chain) -> dict:
        """Per-instance detail of one request: elig, hit, W, rho, tpot, ttft,
        inC, inT (zero where not capacity-eligible) and the choice."""
        ch, cp = _c(chain, np.uint64)
        n = self.n_inst
        out = dict(elig=np.zeros(n, np.uint8), hit=np.zeros(n, np.uint32),
                   W=np.zeros(n), rho=np.zeros(n), tpot=np.zeros(n), ttft=np.zeros(n),
                   inC=np.zeros(n, np.uint8), inT=np.zeros(n, np.uint8))
        out["choice"] = _load().orc_explain(
            self._h, ctypes.byref(model), cp, len(ch),
            *[out[k].ctypes.data for k in ("elig", "hit", "W", "rho", "tpot", "ttft", "inC", "inT")])
        return out

    # conveniences over a generated window
    def window_hits(self, win, nthreads=0):
        return self.hits(win.pool, win.pre_off, win.pre_len, win.tail_off, win.tail_len, nthreads)

    def window_score(self, win, nthreads=0, **policy) -> Decisions:
        return self.score(model_of(win, **policy), win.pool, win.pre_off, win.pre_len,
                          win.tail_off, win.tail_len, nthreads)

    def window_schedule(self, win, follow=None, **policy):
        return self.schedule(model_of(win, **policy), win.pool, win.pre_off, win.pre_len,
                             win.tail_off, win.tail_len, follow=follow)

    def window_replay(self, win, inst, **policy):
        return self.replay(model_of(win, **policy), win.pool, win.pre_off, win.pre_len,
                           win.tail_off, win.tail_len, inst)


def feedback_decode(model: Model, batch, ctx_tok, measured) -> None:
    """EMA calibration of the model's decode factors (in place)."""
    b_, bp = _c(batch, np.int32)
    c_, cp = _c(ctx_tok, np.int64)
    m_, mp = _c(measured, np.float64)
    _load().orc_feedback_decode(ctypes.byref(model), bp, cp, mp, len(b_))


def max_threads() -> int:
    return int(_load().orc_max_threads())
