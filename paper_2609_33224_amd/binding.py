"""ctypes binding of ``libpackserve.so`` (the C ABI in include/packserve.h).

Argument marshalling only: every step of the scoring path runs in the HIP
kernels of the library.  The functions keep the C names.  Device-side calls
take torch CUDA tensors (torch supplies device memory and streams and
nothing else).  There is no CPU fallback: if the library is missing the
import fails.

torch is imported before the library is opened so that both bind to the
same HIP runtime in this process.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch  # noqa: F401  (first: the library must bind to torch's HIP runtime)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpackserve.so")

PS_OK, PS_E_INVAL, PS_E_NOMEM, PS_E_DEVICE, PS_E_STATE, PS_E_RANGE = 0, -1, -2, -3, -4, -5
PS_MAX_SEG = 32
PS_MAX_INST = 65536
PS_MAX_DQ = 4095
PS_MAX_CHAIN = (1 << 24) - 1
PS_F_TTFT_ADMIT, PS_F_NO_KVC_FILTER, PS_F_NO_TPOT_FILTER, PS_F_FALLBACK_DCQ = 1, 2, 4, 8
(PS_SEL_DCQ, PS_SEL_D, PS_SEL_DQ, PS_SEL_DC, PS_SEL_DQC, PS_SEL_HCQ, PS_SEL_RANDOM,
 PS_SEL_LMETRIC) = range(8)


def PS_F_SELECTOR(sel: int) -> int:
    return (int(sel) & 0xF) << 8


PS_R_REJECT, PS_R_FALLBACK, PS_R_TTFT_MISS, PS_R_INVALID = 1, 2, 4, 8

# struct ps_req (24 bytes) and struct ps_result (20 bytes)
PS_REQ_DTYPE = np.dtype([("pre_off", "<i8"), ("tail_off", "<i8"), ("pre_len", "<i4"),
                         ("tail_len", "<i4")])
PS_RESULT_DTYPE = np.dtype([("instance", "<i4"), ("hit_blocks", "<i4"), ("ttft", "<f4"),
                            ("tpot", "<f4"), ("flags", "<u4")])
PS_EVENT_DTYPE = np.dtype([("instance", "<i4"), ("kind", "<i4"), ("tokens", "<i8")])
assert PS_REQ_DTYPE.itemsize == 24 and PS_RESULT_DTYPE.itemsize == 20
assert PS_EVENT_DTYPE.itemsize == 16
PS_EV_PREFILL_DONE, PS_EV_DECODE_TOKENS, PS_EV_FINISHED = 1, 2, 3
PS_LOUT_WINDOW = 1024


class PsModel(ctypes.Structure):
    _fields_ = [
        ("alpha", ctypes.c_float * 6),
        ("n_seg", ctypes.c_int32),
        ("seg_ub", ctypes.c_int32 * PS_MAX_SEG),
        ("beta", (ctypes.c_float * 3) * PS_MAX_SEG),
        ("gamma", ctypes.c_float * PS_MAX_SEG),
        ("eta", ctypes.c_float), ("tpot_slo", ctypes.c_float),
        ("ttft_floor", ctypes.c_float), ("lout", ctypes.c_float),
        ("block_tokens", ctypes.c_int32), ("b_max", ctypes.c_int32),
        ("kv_cap_tokens", ctypes.c_int64),
        ("flags", ctypes.c_uint32),
        ("rand_seed", ctypes.c_uint64),
    ]


class PsInstances(ctypes.Structure):
    _fields_ = [
        ("n_inst", ctypes.c_int32), ("table_cap_blocks", ctypes.c_int32),
        ("blk_off", ctypes.c_void_p), ("blk", ctypes.c_void_p),
        ("decoding", ctypes.c_void_p), ("queued", ctypes.c_void_p),
        ("pending_tok", ctypes.c_void_p), ("ctx_tok", ctypes.c_void_p),
    ]


class PackServeError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"packserve error {code}: {msg}")
        self.code = code


_lib = None


def load_library() -> ctypes.CDLL:
    """Open libpackserve.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "ps_create": ([ctypes.c_int, ctypes.POINTER(vp)], i32),
        "ps_destroy": ([vp], i32),
        "ps_load_instances": ([vp, ctypes.POINTER(PsInstances), ctypes.POINTER(PsModel)], i32),
        "ps_score_window": ([vp, vp, i64, vp, i32, vp], i32),
        "ps_score_window_dev": ([vp, vp, i64, vp, i32, vp, vp, vp], i32),
        "ps_score_window_dev_fixed": ([vp, vp, i64, vp, i32, vp, vp, vp], i32),
        "ps_probe_hits_dev": ([vp, vp, i64, vp, i32, vp, vp], i32),
        "ps_commit": ([vp, vp, i64, vp, vp, i32, ctypes.POINTER(i64)], i32),
        "ps_schedule_window_dev": ([vp, vp, i64, vp, i32, vp, vp, ctypes.POINTER(i64), vp], i32),
        "ps_replay_window_dev": ([vp, vp, i64, vp, i32, vp, vp, ctypes.POINTER(i64), vp], i32),
        "ps_set_schedule_budget": ([vp, i64], i32),
        "ps_set_schedule_speculation": ([vp, i32], i32),
        "ps_read_schedule_stats": ([vp, ctypes.POINTER(i64), ctypes.POINTER(i64)], i32),
        "ps_read_state": ([vp, vp, vp, vp, vp, vp], i32),
        "ps_table_info": ([vp, ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i32)], i32),
        "ps_last_error": ([vp], ctypes.c_char_p),
        "ps_build_id": ([], ctypes.c_char_p),
        "ps_apply_events": ([vp, vp, i32], i32),
        "ps_feedback_decode": ([vp, vp, vp, vp, i32], i32),
        "ps_feedback_output": ([vp, vp, i32], i32),
        "ps_read_model": ([vp, vp, vp, vp], i32),
        "ps_set_timing": ([vp, i32], i32),
        "ps_read_kernel_timing": ([vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_float)], i32),
        "ps_read_timing": ([vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_float),
                            ctypes.POINTER(ctypes.c_float)], i32),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _check(ctx, code):
    if code != PS_OK:
        msg = load_library().ps_last_error(ctx)
        raise PackServeError(code, msg.decode() if msg else "")


def _ptr(a: np.ndarray, dtype) -> tuple:
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def _dev_ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return t.data_ptr()


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


# ------------------------------------------------------------------ structs
def make_model(alpha, seg_ub, beta, gamma, eta, tpot_slo, ttft_floor, lout, block_tokens,
               b_max, kv_cap_tokens, flags=0, rand_seed=0) -> PsModel:
    m = PsModel()
    for k in range(6):
        m.alpha[k] = float(alpha[k])
    m.n_seg = len(seg_ub)
    for s in range(len(seg_ub)):
        m.seg_ub[s] = int(seg_ub[s])
        for k in range(3):
            m.beta[s][k] = float(beta[s][k])
        m.gamma[s] = float(gamma[s])
    m.eta, m.tpot_slo, m.ttft_floor, m.lout = float(eta), float(tpot_slo), float(ttft_floor), float(lout)
    m.block_tokens, m.b_max = int(block_tokens), int(b_max)
    m.kv_cap_tokens, m.flags = int(kv_cap_tokens), int(flags)
    m.rand_seed = int(rand_seed) & 0xFFFFFFFFFFFFFFFF
    return m


def pack_reqs(pre_off, pre_len, tail_off, tail_len) -> np.ndarray:
    r = np.zeros(len(pre_off), dtype=PS_REQ_DTYPE)
    r["pre_off"], r["pre_len"] = pre_off, pre_len
    r["tail_off"], r["tail_len"] = tail_off, tail_len
    return r


# ------------------------------------------------------------------ entry points
def ps_create(device: int = 0) -> ctypes.c_void_p:
    lib = load_library()
    h = ctypes.c_void_p()
    _check(None, lib.ps_create(int(device), ctypes.byref(h)))
    return h


def ps_destroy(ctx) -> None:
    load_library().ps_destroy(ctx)


def ps_last_error(ctx) -> str:
    msg = load_library().ps_last_error(ctx)
    return msg.decode() if msg else ""


def ps_build_id() -> str:
    """Source hash the library was built from (build.source_hash() of a fresh build)."""
    return load_library().ps_build_id().decode()


def ps_load_instances(ctx, n_inst, table_cap_blocks, blk_off, blk, decoding, queued,
                      pending_tok, ctx_tok, model: PsModel) -> None:
    keep = [_ptr(blk_off, np.int64), _ptr(blk, np.uint64), _ptr(decoding, np.int32),
            _ptr(queued, np.int32), _ptr(pending_tok, np.int64), _ptr(ctx_tok, np.int64)]
    inst = PsInstances(int(n_inst), int(table_cap_blocks), *[k[1] for k in keep])
    _check(ctx, load_library().ps_load_instances(ctx, ctypes.byref(inst), ctypes.byref(model)))


def ps_score_window(ctx, pool: np.ndarray, reqs: np.ndarray) -> np.ndarray:
    pool, pp = _ptr(pool, np.uint64)
    reqs = np.ascontiguousarray(reqs, dtype=PS_REQ_DTYPE)
    out = np.zeros(len(reqs), dtype=PS_RESULT_DTYPE)
    _check(ctx, load_library().ps_score_window(ctx, pp, len(pool), reqs.ctypes.data, len(reqs),
                                               out.ctypes.data))
    return out


def ps_score_window_dev(ctx, d_pool: torch.Tensor, pool_len: int, d_reqs: torch.Tensor,
                        n_req: int, d_out: torch.Tensor, d_sizes: Optional[torch.Tensor] = None,
                        stream=None) -> None:
    _check(ctx, load_library().ps_score_window_dev(
        ctx, _dev_ptr(d_pool), int(pool_len), _dev_ptr(d_reqs), int(n_req), _dev_ptr(d_out),
        _dev_ptr(d_sizes), _stream_handle(stream)))


def ps_score_window_dev_fixed(ctx, d_pool: torch.Tensor, pool_len: int, d_reqs: torch.Tensor,
                              n_req: int, d_out: torch.Tensor,
                              d_sizes: Optional[torch.Tensor] = None, stream=None) -> None:
    """ps_score_window_dev with the group table in the library's fixed device
    array (no allocation; at most 65,536 requests per call)."""
    _check(ctx, load_library().ps_score_window_dev_fixed(
        ctx, _dev_ptr(d_pool), int(pool_len), _dev_ptr(d_reqs), int(n_req), _dev_ptr(d_out),
        _dev_ptr(d_sizes), _stream_handle(stream)))


def ps_probe_hits_dev(ctx, d_pool: torch.Tensor, pool_len: int, d_reqs: torch.Tensor,
                      n_req: int, d_hits: torch.Tensor, stream=None) -> None:
    _check(ctx, load_library().ps_probe_hits_dev(
        ctx, _dev_ptr(d_pool), int(pool_len), _dev_ptr(d_reqs), int(n_req), _dev_ptr(d_hits),
        _stream_handle(stream)))


def ps_schedule_window_dev(ctx, d_pool: torch.Tensor, pool_len: int, d_reqs: torch.Tensor,
                           n_req: int, d_out: torch.Tensor,
                           d_sizes: Optional[torch.Tensor] = None, stream=None) -> int:
    """Algorithm 1 per arrival over a device-resident window; returns the
    number of blocks refused at the table cap."""
    dropped = ctypes.c_int64()
    _check(ctx, load_library().ps_schedule_window_dev(
        ctx, _dev_ptr(d_pool), int(pool_len), _dev_ptr(d_reqs), int(n_req), _dev_ptr(d_out),
        _dev_ptr(d_sizes), ctypes.byref(dropped), _stream_handle(stream)))
    return int(dropped.value)


def ps_replay_window_dev(ctx, d_pool: torch.Tensor, pool_len: int, d_reqs: torch.Tensor,
                         n_req: int, d_inst: torch.Tensor, d_out: torch.Tensor,
                         stream=None) -> int:
    """Latencies of given placements at their arrival, committing each;
    returns the number of blocks refused at the table cap."""
    dropped = ctypes.c_int64()
    _check(ctx, load_library().ps_replay_window_dev(
        ctx, _dev_ptr(d_pool), int(pool_len), _dev_ptr(d_reqs), int(n_req), _dev_ptr(d_inst),
        _dev_ptr(d_out), ctypes.byref(dropped), _stream_handle(stream)))
    return int(dropped.value)


def ps_commit(ctx, pool: np.ndarray, reqs: np.ndarray, inst: np.ndarray) -> int:
    pool, pp = _ptr(pool, np.uint64)
    reqs = np.ascontiguousarray(reqs, dtype=PS_REQ_DTYPE)
    inst, ip = _ptr(inst, np.int32)
    dropped = ctypes.c_int64()
    _check(ctx, load_library().ps_commit(ctx, pp, len(pool), reqs.ctypes.data, ip, len(inst),
                                         ctypes.byref(dropped)))
    return int(dropped.value)


def ps_read_state(ctx, n_inst: int) -> dict:
    out = dict(D=np.zeros(n_inst, np.int32), Q=np.zeros(n_inst, np.int32),
               P=np.zeros(n_inst, np.int64), S=np.zeros(n_inst, np.int64),
               set_size=np.zeros(n_inst, np.int64))
    _check(ctx, load_library().ps_read_state(ctx, *[out[k].ctypes.data for k in
                                                    ("D", "Q", "P", "S", "set_size")]))
    return out


def ps_table_info(ctx) -> dict:
    slots, nbytes, lds = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
    _check(ctx, load_library().ps_table_info(ctx, ctypes.byref(slots), ctypes.byref(nbytes),
                                             ctypes.byref(lds)))
    return dict(slots_per_table=slots.value, table_bytes=nbytes.value,
                hits_in_lds=bool(lds.value))


def ps_apply_events(ctx, inst, kind, tokens) -> None:
    ev = np.zeros(len(inst), dtype=PS_EVENT_DTYPE)
    ev["instance"], ev["kind"], ev["tokens"] = inst, kind, tokens
    _check(ctx, load_library().ps_apply_events(ctx, ev.ctypes.data, len(ev)))


def ps_feedback_decode(ctx, batch, ctx_tok, measured_s) -> None:
    b, bp = _ptr(batch, np.int32)
    c, cp = _ptr(ctx_tok, np.int64)
    m, mp = _ptr(measured_s, np.float32)
    _check(ctx, load_library().ps_feedback_decode(ctx, bp, cp, mp, len(b)))


def ps_feedback_output(ctx, out_len) -> None:
    o, op = _ptr(out_len, np.int32)
    _check(ctx, load_library().ps_feedback_output(ctx, op, len(o)))


def ps_read_model(ctx) -> dict:
    g = np.zeros(PS_MAX_SEG, np.float32)
    lout = ctypes.c_float()
    n = ctypes.c_int32()
    _check(ctx, load_library().ps_read_model(ctx, g.ctypes.data, ctypes.byref(lout),
                                             ctypes.byref(n)))
    return dict(gamma=g[:n.value].copy(), lout=float(lout.value))


# ------------------------------------------------------------------ tensors
def to_device_u64(a: np.ndarray, device="cuda") -> torch.Tensor:
    """uint64 host array -> int64 device tensor holding the same bits."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(device)


def to_device_bytes(a: np.ndarray, device="cuda") -> torch.Tensor:
    """Structured host array -> uint8 device tensor of its bytes."""
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.uint8).reshape(-1).copy()).to(device)


def results_from_device(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(PS_RESULT_DTYPE).copy()


class Scorer:
    """Owns one context; the methods forward to the C entry points."""

    def __init__(self, device: int = 0):
        self.ctx = ps_create(device)
        self.n_inst = 0

    def close(self):
        if self.ctx:
            ps_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load(self, n_inst, cap, blk_off, blk, D, Q, P, S, model: PsModel):
        ps_load_instances(self.ctx, n_inst, cap, blk_off, blk, D, Q, P, S, model)
        self.n_inst = int(n_inst)

    def score(self, pool, reqs) -> np.ndarray:
        return ps_score_window(self.ctx, pool, reqs)

    def score_dev(self, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes=None, stream=None):
        ps_score_window_dev(self.ctx, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes, stream)

    def score_dev_fixed(self, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes=None, stream=None):
        ps_score_window_dev_fixed(self.ctx, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes, stream)

    def set_timing(self, on: bool) -> None:
        _check(self.ctx, load_library().ps_set_timing(self.ctx, 1 if on else 0))

    def read_timing(self) -> tuple:
        """(calls, mean ms of the prefix-group pass, mean ms of the scoring
        kernel) over the scoring calls timed since the last read."""
        n, g, k = ctypes.c_int32(), ctypes.c_float(), ctypes.c_float()
        _check(self.ctx, load_library().ps_read_timing(self.ctx, ctypes.byref(n), ctypes.byref(g),
                                                       ctypes.byref(k)))
        return int(n.value), float(g.value), float(k.value)

    def read_kernel_timing(self) -> tuple:
        """(calls, [mean ms of the claim pass, group walk, lean scorer,
        general scorer]) over the scoring calls timed since the last read."""
        n = ctypes.c_int32()
        ms = (ctypes.c_float * 4)()
        _check(self.ctx, load_library().ps_read_kernel_timing(self.ctx, ctypes.byref(n), ms))
        return int(n.value), [float(x) for x in ms]

    def hits_dev(self, d_pool, pool_len, d_reqs, n_req, d_hits, stream=None):
        ps_probe_hits_dev(self.ctx, d_pool, pool_len, d_reqs, n_req, d_hits, stream)

    def commit(self, pool, reqs, inst) -> int:
        return ps_commit(self.ctx, pool, reqs, inst)

    def schedule_dev(self, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes=None, stream=None) -> int:
        return ps_schedule_window_dev(self.ctx, d_pool, pool_len, d_reqs, n_req, d_out, d_sizes,
                                      stream)

    def set_schedule_budget(self, n_bytes: int) -> None:
        _check(self.ctx, load_library().ps_set_schedule_budget(self.ctx, int(n_bytes)))

    def set_schedule_speculation(self, batch: int) -> None:
        _check(self.ctx, load_library().ps_set_schedule_speculation(self.ctx, int(batch)))

    def schedule_stats(self) -> tuple:
        """(decided from speculation, scored in full) of the last schedule call."""
        a, b = ctypes.c_int64(), ctypes.c_int64()
        _check(self.ctx, load_library().ps_read_schedule_stats(self.ctx, ctypes.byref(a),
                                                                ctypes.byref(b)))
        return int(a.value), int(b.value)

    def replay_dev(self, d_pool, pool_len, d_reqs, n_req, d_inst, d_out, stream=None) -> int:
        return ps_replay_window_dev(self.ctx, d_pool, pool_len, d_reqs, n_req, d_inst, d_out, stream)

    def state(self) -> dict:
        return ps_read_state(self.ctx, self.n_inst)

    def table_info(self) -> dict:
        return ps_table_info(self.ctx)

    def apply_events(self, inst, kind, tokens) -> None:
        ps_apply_events(self.ctx, inst, kind, tokens)

    def feedback_decode(self, batch, ctx_tok, measured_s) -> None:
        ps_feedback_decode(self.ctx, batch, ctx_tok, measured_s)

    def feedback_output(self, out_len) -> None:
        ps_feedback_output(self.ctx, out_len)

    def model(self) -> dict:
        return ps_read_model(self.ctx)
