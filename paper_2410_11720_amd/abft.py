"""ctypes binding of libattn_abft.so (include/attn_abft.h).

Argument marshalling only: every step of the protected layer runs in the
HIP library. torch tensors provide device memory and the current stream;
their data pointers are passed through the C ABI unchanged. If the built
library is missing, importing this module raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libattn_abft.so")

OPS = ("Q", "K", "V", "AS", "CL", "O", "dCL", "dWO", "dAP", "dV", "dQ", "dK",
       "dWQ", "dWK", "dWV", "dX")
OP_ID = {n: i for i, n in enumerate(OPS)}
KINDS = ("NUMERIC", "NEAR_INF", "INF", "NAN", "-")
ACTIONS = ("RECOMPUTE", "DELTA", "RECONSTRUCT", "UNCORRECTABLE")

ABFT_OK = 0
BF16, FP32 = 0, 1
SEC_AS, SEC_CL, SEC_O, SEC_BWD, SEC_ALL = 1, 2, 4, 8, 15
FLAG_ROOT_CHECK, FLAG_REPORT_APPEND, FLAG_UNPROTECTED, FLAG_FUSED = 1, 2, 4, 8

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      f"(or python -m paper_2410_11720_amd._build)")
_lib = ctypes.CDLL(LIB_PATH)


class Config(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seq", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("heads", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("causal", ctypes.c_int32),
                ("block_rows", ctypes.c_int32), ("scale", ctypes.c_float),
                ("t_near_inf", ctypes.c_float), ("t_correct", ctypes.c_float),
                ("e_rel", ctypes.c_float), ("sections", ctypes.c_uint32),
                ("flags", ctypes.c_uint32)]


FAULT_SET, FAULT_FLIP = 0, 1


class Fault(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("b", ctypes.c_int32), ("h", ctypes.c_int32),
                ("row", ctypes.c_int32), ("col", ctypes.c_int32), ("value", ctypes.c_float),
                ("mode", ctypes.c_int32)]


class Event(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("b", ctypes.c_int32), ("h", ctypes.c_int32),
                ("row", ctypes.c_int32), ("col", ctypes.c_int32), ("kind", ctypes.c_int32),
                ("action", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("observed", ctypes.c_float), ("reserved2", ctypes.c_float)]


class FreqOp(ctypes.Structure):
    _fields_ = [("flops", ctypes.c_double), ("p", ctypes.c_double * 3)]


class FreqSection(ctypes.Structure):
    _fields_ = [("n_ops", ctypes.c_int32), ("first_op", ctypes.c_int32),
                ("cost", ctypes.c_double)]


REPORT_HEADER = 32  # bytes before the event array
assert ctypes.sizeof(Event) == 40 and ctypes.sizeof(Fault) == 28

_vp, _sz, _i32, _i64, _f32, _u32 = (ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32,
                                   ctypes.c_int64, ctypes.c_float, ctypes.c_uint32)
_P = ctypes.POINTER(Config)
_sig = {
    "attn_abft_workspace_bytes": (_sz, [_P]),
    "attn_abft_report_bytes": (_sz, [_i32]),
    "attn_abft_report_init": (ctypes.c_int, [_vp, _i32, _vp]),
    "attn_abft_forward": (ctypes.c_int, [_P, _vp, _vp, _vp, _vp, _vp, _sz, _vp, _i32, _vp, _vp]),
    "attn_abft_backward": (ctypes.c_int, [_P, _vp, _vp, _vp, _vp, _vp, _sz, _vp, _vp, _vp,
                                          _vp, _i32, _vp, _vp]),
    "attn_abft_forward_stages": (ctypes.c_int, [_P, _vp, _vp, _vp, _vp, _vp, _sz, _vp, _i32, _vp,
                                                _u32, _vp]),
    "attn_abft_backward_stages": (ctypes.c_int, [_P, _vp, _vp, _vp, _vp, _vp, _sz, _vp, _vp, _vp,
                                                 _vp, _i32, _vp, _u32, _vp]),
    "encode_checksums": (ctypes.c_int, [_vp, _i32, _i64, _i64, _i64, _i64, _i64, _i32, _i32,
                                        _vp, _vp, _vp]),
    "verify_and_correct": (ctypes.c_int, [_vp, _i32, _i64, _i64, _i64, _i64, _i64, _i32, _i32,
                                          _vp, _vp, _f32, _f32, _f32, _i32, _vp, _vp]),
    "attn_abft_workspace_offsets": (ctypes.c_int, [_P, ctypes.POINTER(_sz),
                                                   ctypes.POINTER(_sz), ctypes.POINTER(_sz)]),
    "attn_abft_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "attn_abft_workspace_tensor": (ctypes.c_int, [_P, _i32, ctypes.POINTER(_sz)]),
    "attn_abft_unsafe_probability": (ctypes.c_int, [ctypes.POINTER(FreqOp),
                                                    ctypes.POINTER(FreqSection), _i32, _vp,
                                                    _vp, _vp]),
    "attn_abft_optimize_frequencies": (ctypes.c_int, [ctypes.POINTER(FreqOp),
                                                      ctypes.POINTER(FreqSection), _i32, _vp,
                                                      ctypes.c_double, _vp]),
    "attn_abft_sections_for_step": (_u32, [_vp, _i64]),
    "attn_abft_forward_noalloc": (ctypes.c_int, [_P, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp]),
}
for _name, (_res, _args) in _sig.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


class AbftError(RuntimeError):
    pass


def strerror(status: int) -> str:
    return _lib.attn_abft_strerror(status).decode()


def _check(status: int, what: str):
    if status != ABFT_OK:
        raise AbftError(f"{what}: {strerror(status)} ({status})")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


@dataclasses.dataclass
class LayerConfig:
    batch: int
    seq: int
    hidden: int
    heads: int
    dtype: str = "bf16"          # "bf16" | "f32"
    causal: bool = False
    block_rows: int = 128
    scale: float = 0.0
    t_near_inf: float = 1e10
    t_correct: float = 1e5
    e_rel: float = 0.0
    sections: int = SEC_ALL
    root_check: bool = True
    protect: bool = True
    fused: bool = False          # forward attention core in one kernel (no AS/AP)

    def to_c(self, append=False) -> Config:
        flags = (FLAG_ROOT_CHECK if self.root_check else 0)
        flags |= (FLAG_REPORT_APPEND if append else 0)
        flags |= (0 if self.protect else FLAG_UNPROTECTED)
        flags |= (FLAG_FUSED if self.fused else 0)
        return Config(self.batch, self.seq, self.hidden, self.heads,
                      FP32 if self.dtype == "f32" else BF16, int(self.causal), self.block_rows,
                      self.scale, self.t_near_inf, self.t_correct, self.e_rel, self.sections,
                      flags)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


def attn_abft_workspace_bytes(cfg: LayerConfig) -> int:
    c = cfg.to_c()
    n = _lib.attn_abft_workspace_bytes(ctypes.byref(c))
    if n == 0:
        raise AbftError("invalid configuration")
    return n


def attn_abft_report_bytes(capacity: int) -> int:
    return _lib.attn_abft_report_bytes(capacity)


def attn_abft_report_init(report, capacity, stream=None):
    _check(_lib.attn_abft_report_init(_ptr(report), capacity, _stream(stream)), "report_init")


def attn_abft_workspace_offsets(cfg: LayerConfig):
    c = cfg.to_c()
    q, a, l = _sz(), _sz(), _sz()
    _check(_lib.attn_abft_workspace_offsets(ctypes.byref(c), ctypes.byref(q), ctypes.byref(a),
                                            ctypes.byref(l)), "workspace_offsets")
    return q.value, a.value, l.value


def attn_abft_forward(cfg: LayerConfig, X, Wqkv, Wo, O, workspace, faults, n_faults, report,
                      stream=None, append=False):
    c = cfg.to_c(append)
    _check(_lib.attn_abft_forward(ctypes.byref(c), _ptr(X), _ptr(Wqkv), _ptr(Wo), _ptr(O),
                                  _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _ptr(faults), n_faults, _ptr(report), _stream(stream)),
           "attn_abft_forward")


def attn_abft_forward_noalloc(cfg: LayerConfig, X, Wqkv, Wo, O, faults, n_faults, report,
                              stream=None, append=False):
    c = cfg.to_c(append)
    _check(_lib.attn_abft_forward_noalloc(ctypes.byref(c), _ptr(X), _ptr(Wqkv), _ptr(Wo), _ptr(O),
                                          _ptr(faults), n_faults, _ptr(report), _stream(stream)),
           "attn_abft_forward_noalloc")


def attn_abft_backward(cfg: LayerConfig, dO, X, Wqkv, Wo, workspace, dX, dWqkv, dWo, faults,
                       n_faults, report, stream=None, append=False):
    c = cfg.to_c(append)
    _check(_lib.attn_abft_backward(ctypes.byref(c), _ptr(dO), _ptr(X), _ptr(Wqkv), _ptr(Wo),
                                   _ptr(workspace), workspace.numel() * workspace.element_size(),
                                   _ptr(dX), _ptr(dWqkv), _ptr(dWo), _ptr(faults), n_faults,
                                   _ptr(report), _stream(stream)), "attn_abft_backward")


STAGE_ALL = 0x7FF
FWD_STAGES = {"encode": 0x001, "qkv": 0x002, "score": 0x004, "softmax": 0x008,
              "context": 0x010, "out": 0x020}
BWD_STAGES = {"encode": 0x001, "dCL": 0x002, "dWo": 0x004, "dAP": 0x008, "dV": 0x010,
              "softmax_bwd": 0x020, "dQ": 0x040, "dK": 0x080, "dWqkv": 0x100, "dX": 0x200}


def attn_abft_forward_stages(cfg: LayerConfig, X, Wqkv, Wo, O, workspace, faults, n_faults,
                             report, stages, stream=None, append=False):
    c = cfg.to_c(append)
    _check(_lib.attn_abft_forward_stages(ctypes.byref(c), _ptr(X), _ptr(Wqkv), _ptr(Wo), _ptr(O),
                                         _ptr(workspace),
                                         workspace.numel() * workspace.element_size(),
                                         _ptr(faults), n_faults, _ptr(report), stages,
                                         _stream(stream)), "attn_abft_forward_stages")


def attn_abft_backward_stages(cfg: LayerConfig, dO, X, Wqkv, Wo, workspace, dX, dWqkv, dWo,
                              faults, n_faults, report, stages, stream=None, append=False):
    c = cfg.to_c(append)
    _check(_lib.attn_abft_backward_stages(ctypes.byref(c), _ptr(dO), _ptr(X), _ptr(Wqkv),
                                          _ptr(Wo), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(),
                                          _ptr(dX), _ptr(dWqkv), _ptr(dWo), _ptr(faults),
                                          n_faults, _ptr(report), stages, _stream(stream)),
           "attn_abft_backward_stages")


def encode_checksums(A, dtype, batch, rows, cols, ld, batch_stride, block_rows, block_cols,
                     col_chk, row_chk, stream=None):
    _check(_lib.encode_checksums(_ptr(A), dtype, batch, rows, cols, ld, batch_stride,
                                 block_rows, block_cols, _ptr(col_chk), _ptr(row_chk),
                                 _stream(stream)), "encode_checksums")


def verify_and_correct(C, dtype, batch, rows, cols, ld, batch_stride, block_rows, block_cols,
                       col_chk, row_chk, t_near_inf, t_correct, e_rel, op_tag, report,
                       stream=None):
    _check(_lib.verify_and_correct(_ptr(C), dtype, batch, rows, cols, ld, batch_stride,
                                   block_rows, block_cols, _ptr(col_chk), _ptr(row_chk),
                                   t_near_inf, t_correct, e_rel, op_tag, _ptr(report),
                                   _stream(stream)), "verify_and_correct")


# ---- conveniences for callers holding torch tensors -----------------------

def _freq_args(sections):
    """sections: [(cost, [(flops, (p_inf, p_nan, p_ninf)), ...]), ...]"""
    ops, secs = [], []
    for cost, sec_ops in sections:
        secs.append(FreqSection(len(sec_ops), len(ops), float(cost)))
        for flops, p in sec_ops:
            ops.append(FreqOp(float(flops), (ctypes.c_double * 3)(*[float(x) for x in p])))
    oa = (FreqOp * max(1, len(ops)))(*ops)
    sa = (FreqSection * len(secs))(*secs)
    return oa, sa, len(secs)


def _doubles(xs):
    return (ctypes.c_double * len(xs))(*[float(x) for x in xs])


def attn_abft_unsafe_probability(sections, lam, freqs) -> float:
    oa, sa, n = _freq_args(sections)
    out = ctypes.c_double()
    _check(_lib.attn_abft_unsafe_probability(oa, sa, n, _doubles(lam), _doubles(freqs),
                                             ctypes.byref(out)), "unsafe_probability")
    return out.value


def attn_abft_optimize_frequencies(sections, lam, fail_target) -> list:
    oa, sa, n = _freq_args(sections)
    out = (ctypes.c_double * n)()
    _check(_lib.attn_abft_optimize_frequencies(oa, sa, n, _doubles(lam), float(fail_target),
                                               out), "optimize_frequencies")
    return list(out)


def attn_abft_sections_for_step(freqs4, step: int) -> int:
    return int(_lib.attn_abft_sections_for_step(_doubles(freqs4), int(step)))


def faults_to_device(faults, device="cuda"):
    """Pack (op, b, h, row, col, value[, mode]) tuples into a device array
    of abft_fault records; mode "set" (default) or "flip". Returns (tensor
    or None, count)."""
    faults = [f.as_tuple() if hasattr(f, "as_tuple") else tuple(f) for f in faults]
    if not faults:
        return None, 0

    def rec(t):
        o, b, h, r, c, v = t[:6]
        mode = FAULT_FLIP if len(t) > 6 and t[6] == "flip" else FAULT_SET
        return Fault(OP_ID[o] if isinstance(o, str) else int(o), b, h, r, c, float(v), mode)
    arr = (Fault * len(faults))(*[rec(t) for t in faults])
    host = torch.frombuffer(bytearray(bytes(arr)), dtype=torch.uint8)
    return host.to(device), len(faults)


def new_report(capacity=4096, device="cuda", stream=None):
    rep = torch.empty(attn_abft_report_bytes(capacity), dtype=torch.uint8, device=device)
    attn_abft_report_init(rep, capacity, stream)
    return rep


def read_report(report) -> dict:
    """Copy a report to the host: counters and the event list as tuples
    (op, b, h, row, col, kind, action)."""
    raw = bytes(report.cpu().numpy().tobytes())
    n_events, n_corr, n_unc, cap, overflow = (int.from_bytes(raw[4 * i:4 * i + 4], "little",
                                                             signed=True) for i in range(5))
    evs = []
    for k in range(min(n_events, cap)):
        e = Event.from_buffer_copy(raw, REPORT_HEADER + k * ctypes.sizeof(Event))
        evs.append((OPS[e.op], e.b, e.h, e.row, e.col, KINDS[e.kind], ACTIONS[e.action]))
    return dict(n_events=n_events, n_corrected=n_corr, n_uncorrectable=n_unc,
                capacity=cap, overflow=overflow, events=evs)


class ProtectedAttention:
    """Owns the workspace and report of one layer shape and runs the
    protected forward and backward through the C ABI."""

    def __init__(self, cfg: LayerConfig, device="cuda", capacity=4096):
        self.cfg = cfg
        self.device = device
        self.workspace = torch.empty(attn_abft_workspace_bytes(cfg), dtype=torch.uint8,
                                     device=device)
        self.report = new_report(capacity, device)
        self.report_bwd = new_report(capacity, device)

    def forward(self, X, Wqkv, Wo, faults=None, O=None):
        c = self.cfg
        if O is None:
            O = torch.empty((c.batch, c.seq, c.hidden), dtype=c.torch_dtype, device=self.device)
        f, n = faults if faults is not None else (None, 0)
        attn_abft_forward(c, X, Wqkv, Wo, O, self.workspace, f, n, self.report)
        return O

    def backward(self, dO, X, Wqkv, Wo, faults=None, dX=None, dWqkv=None, dWo=None):
        c = self.cfg
        if dX is None:
            dX = torch.empty((c.batch, c.seq, c.hidden), dtype=c.torch_dtype, device=self.device)
        if dWqkv is None:
            dWqkv = torch.empty((c.hidden, 3 * c.hidden), dtype=torch.float32, device=self.device)
        if dWo is None:
            dWo = torch.empty((c.hidden, c.hidden), dtype=torch.float32, device=self.device)
        f, n = faults if faults is not None else (None, 0)
        attn_abft_backward(c, dO, X, Wqkv, Wo, self.workspace, dX, dWqkv, dWo, f, n,
                           self.report_bwd)
        return dX, dWqkv, dWo

    TENSORS = ("QKV", "AS", "AP", "CL", "dQKV", "dCL", "APc", "APr", "dAS")

    def tensor(self, which):
        """View of a tensor the forward or backward leaves in the workspace:
        "QKV", "AS" (until the next backward), "AP", "CL", "dQKV", "dCL",
        "dAS" (storage dtype), "APc", "APr" (fp32 checksums of AP)."""
        c = self.cfg
        k = self.TENSORS.index(which)
        off = ctypes.c_size_t()
        _check(_lib.attn_abft_workspace_tensor(ctypes.byref(c.to_c()), k, ctypes.byref(off)),
               "workspace_tensor")
        B, S, H, nh = c.batch, c.seq, c.hidden, c.heads
        nq = S // c.block_rows
        shape = {"QKV": (B, S, 3 * H), "AS": (B, nh, S, S), "AP": (B, nh, S, S),
                 "CL": (B, S, H), "dQKV": (B, S, 3 * H), "dCL": (B, S, H),
                 "dAS": (B, nh, S, S), "APc": (B, nh, nq, 2, S),
                 "APr": (B, nh, S, nq, 2)}[which]
        dt = torch.float32 if which in ("APc", "APr") else c.torch_dtype
        es = 4 if dt == torch.float32 else 2
        n = 1
        for x in shape:
            n *= x
        o = off.value
        return self.workspace[o:o + n * es].view(dt).view(*shape)

    def saved(self):
        """Views of the saved QKV, AP and CL inside the workspace."""
        c = self.cfg
        q, a, l = attn_abft_workspace_offsets(c)
        es = 4 if c.dtype == "f32" else 2
        T, H, S = c.batch * c.seq, c.hidden, c.seq

        def view(off, n, shape):
            return self.workspace[off:off + n * es].view(c.torch_dtype).view(*shape)
        return (view(q, T * 3 * H, (c.batch, S, 3 * H)),
                view(a, c.batch * c.heads * S * S, (c.batch, c.heads, S, S)),
                view(l, T * H, (c.batch, S, H)))
