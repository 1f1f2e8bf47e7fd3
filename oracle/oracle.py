"""WaveRNN oracle -- test infrastructure only.

ctypes wrapper around ``wavernn_oracle.c``: a plain scalar CPU implementation of
the WaveRNN sampling step (Eq. 2 and the dual softmax of Sec. 2, the masked
input matrix I*, the coarse-then-fine order of the Fig. 1 caption).  Only the
tests, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg may use
it.  It shares no code with the GPU library and never imports it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wavernn_oracle.c")
_BUILD = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD, "liborc.so")
_lib = None

N_CLASSES = 256


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (-O2, no fp contraction, no fast-math)."""
    os.makedirs(_BUILD, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < max(
        os.path.getmtime(_SRC), os.path.getmtime(os.path.join(_HERE, "wavernn_oracle.h"))
    ):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-std=c11",
             "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Cnn(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "Rc", "Cc", "Dx", "layers")] + [
        (n, ctypes.POINTER(ctypes.c_float)) for n in ("Win", "bin", "Wc", "bc", "Wo", "bo", "Wp", "bp")]


class _Model(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int32), ("Dc", ctypes.c_int32), ("frame_len", ctypes.c_int32),
                ("B", ctypes.c_int32), ("Dx", ctypes.c_int32), ("F", ctypes.c_int32)] + [
        (n, ctypes.POINTER(ctypes.c_float))
        for n in ("R", "I", "b", "Wc", "Wx", "O1", "b1", "O2", "b2", "O3", "b3", "O4", "b4")] + [
        ("cnn", ctypes.POINTER(_Cnn))]


class _FusedModel(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int32), ("F", ctypes.c_int32), ("Dc", ctypes.c_int32),
                ("frame_len", ctypes.c_int32)] + [
        (n, ctypes.POINTER(ctypes.c_float)) for n in ("R", "I", "b", "Wc", "O1", "b1", "O2", "b2")]


def lib():
    global _lib
    if _lib is None:
        _lib = load(build())
    return _lib


def load(path: str):
    """Load an oracle build (tests load planted-mistake builds this way)."""
    L = ctypes.CDLL(path)
    f32, i32, i64, u64 = ctypes.c_float, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    vp = ctypes.c_void_p
    for name in ("orc_exp", "orc_sigmoid", "orc_tanh"):
        getattr(L, name).restype = f32
        getattr(L, name).argtypes = [f32]
    L.orc_scale.restype = f32
    L.orc_scale.argtypes = [ctypes.c_int]
    L.orc_philox4x64_10.restype = None
    L.orc_philox4x64_10.argtypes = [vp, vp, vp]
    L.orc_uniforms.restype = None
    L.orc_uniforms.argtypes = [u64, u64, i64, ctypes.POINTER(f32), ctypes.POINTER(f32)]
    L.orc_draw.restype = ctypes.c_int
    L.orc_draw.argtypes = [vp, ctypes.c_int, f32]
    L.orc_subscale_context.restype = None
    L.orc_subscale_context.argtypes = [ctypes.POINTER(_Model), vp, i64, i32, i64, vp]
    L.orc_fused_run.restype = ctypes.c_int
    L.orc_fused_run.argtypes = [ctypes.POINTER(_FusedModel), i32, i64, vp, i64, u64, vp, vp, vp, vp, vp, vp]
    L.orc_ctx_cnn.restype = ctypes.c_int
    L.orc_ctx_cnn.argtypes = [ctypes.POINTER(_Cnn), vp, i64, i32, vp]
    L.orc_run_lanes.restype = ctypes.c_int
    L.orc_run_lanes.argtypes = [ctypes.POINTER(_Model), i32, i64, vp, i64, vp, vp, vp, vp, vp, vp, vp, i32, i32]
    L.orc_run.restype = ctypes.c_int
    L.orc_run.argtypes = [ctypes.POINTER(_Model), i32, i64, i64, vp, i64, u64, vp, vp, vp, vp, vp,
                          vp, vp, vp]
    return L


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def exp(y: float) -> float:
    return lib().orc_exp(y)


def sigmoid(x: float) -> float:
    return lib().orc_sigmoid(x)


def tanh(x: float) -> float:
    return lib().orc_tanh(x)


def scale(v: int) -> float:
    return lib().orc_scale(v)


def philox4x64_10(ctr, key):
    c = np.asarray(ctr, dtype=np.uint64).copy()
    k = np.asarray(key, dtype=np.uint64).copy()
    out = np.zeros(4, dtype=np.uint64)
    lib().orc_philox4x64_10(_p(c), _p(k), _p(out))
    return out


def uniforms(seed: int, stream: int, t: int):
    uc, uf = ctypes.c_float(), ctypes.c_float()
    lib().orc_uniforms(seed, stream, t, ctypes.byref(uc), ctypes.byref(uf))
    return uc.value, uf.value


def draw(z, u: float) -> int:
    z = np.ascontiguousarray(z, dtype=np.float32)
    return lib().orc_draw(_p(z), len(z), u)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """fp32 -> nearest bf16 value (ties to even), returned widened to fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    bias = ((bits >> 16) & 1) + 0x7FFF
    r = ((bits + bias) >> 16) << 16
    nan = np.isnan(a)
    out = r.astype(np.uint32).view(np.float32).copy()
    out[nan] = a[nan]
    return out


@dataclass
class Weights:
    """fp32 weights (row-major, gate order u, r, e) as the oracle reads them."""
    H: int
    R: np.ndarray
    I: np.ndarray
    b: np.ndarray
    O1: np.ndarray
    b1: np.ndarray
    O2: np.ndarray
    b2: np.ndarray
    O3: np.ndarray
    b3: np.ndarray
    O4: np.ndarray
    b4: np.ndarray
    Wc: np.ndarray | None = None
    Wx: np.ndarray | None = None
    frame_len: int = 120
    B: int = 1
    F: int = -1          # subscale future horizon (Sec. 4.2); < 0: lockstep rows
    cnn: dict | None = None   # conditioning network (ctx_cnn's keys), replaces the window context

    @staticmethod
    def from_dict(d: dict, bf16: bool = False) -> "Weights":
        keys = ("R", "I", "b", "O1", "b1", "O2", "b2", "O3", "b3", "O4", "b4", "Wc", "Wx")
        kw = {}
        for k in keys:
            v = d.get(k)
            if v is None:
                kw[k] = None
                continue
            v = np.ascontiguousarray(v, dtype=np.float32)
            kw[k] = bf16_round(v) if bf16 else v.copy()
        cnn = d.get("cnn")
        if cnn is not None:
            cnn = dict(cnn, **{k: (bf16_round(cnn[k]) if bf16 else np.ascontiguousarray(cnn[k], np.float32))
                               for k in CNN_KEYS})
        return Weights(H=int(d["H"]), frame_len=int(d.get("frame_len", 120)), B=int(d.get("B", 1)),
                       F=int(d.get("F", -1)), cnn=cnn, **kw)


CNN_KEYS = ("Win", "bin", "Wc", "bc", "Wo", "bo", "Wp", "bp")


def _cnn(w: dict) -> _Cnn:
    """The C view of a conditioning-network dict (arrays must stay alive with it)."""
    keep = {k: np.ascontiguousarray(w[k], np.float32) for k in CNN_KEYS}
    B, L = int(w["B"]), int(w["layers"])
    Rc, Dx = keep["Win"].shape[0], keep["Wp"].shape[0]
    Cc = keep["bc"].shape[1] if L > 0 else 1
    fp = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    c = _Cnn(B, Rc, Cc, Dx, L, *[fp(keep[k]) for k in CNN_KEYS])
    c._keep = keep
    return c


def _model(w: Weights):
    f = ctypes.POINTER(ctypes.c_float)

    def fp(a):
        return ctypes.cast(a.ctypes.data, f) if a is not None else ctypes.cast(None, f)

    m = _Model()
    m.H = w.H
    m.Dc = 0 if w.Wc is None else w.Wc.shape[1]
    m.Dx = 0 if w.Wx is None else w.Wx.shape[1]
    m.frame_len = w.frame_len
    m.B = w.B
    m.F = w.F
    for n in ("R", "I", "b", "Wc", "Wx", "O1", "b1", "O2", "b2", "O3", "b3", "O4", "b4"):
        setattr(m, n, fp(getattr(w, n)))
    if w.cnn is not None:
        c = _cnn(w.cnn)
        m.cnn = ctypes.pointer(c)
        m._cnn = c
    return m


def subscale_context(w: Weights, seq, s: int, i: int) -> np.ndarray:
    """The context vector [Dx] of sample B*i + s of one utterance whose samples are seq [N]."""
    seq = np.ascontiguousarray(seq, np.uint16)
    ctx = np.zeros(w.Wx.shape[1], np.float32)
    m = _model(w)
    lib().orc_subscale_context(ctypes.byref(m), _p(seq), len(seq), s, i, _p(ctx))
    return ctx


def run(w: Weights, S: int, T: int, feat=None, seed: int = 1, target=None, h0=None, c0=None, f0=None,
        t0: int = 0, logits: bool = False, nll: bool = False) -> dict:
    """Sample (target None) or teacher-force S utterances of T samples.

    Returns dict(out [S][T] uint16, h [S*B][H], c, f [S*B] uint8, zc, zf [S][T][256], nll [S][T])."""
    L = lib()
    B = w.B
    H = w.H
    h = np.zeros((S * B, H), np.float32) if h0 is None else np.ascontiguousarray(h0, np.float32).copy()
    c = np.full(S * B, 128, np.uint8) if c0 is None else np.ascontiguousarray(c0, np.uint8).copy()
    f = np.zeros(S * B, np.uint8) if f0 is None else np.ascontiguousarray(f0, np.uint8).copy()
    out = np.zeros((S, T), np.uint16)
    n_frames = 0
    if feat is not None:
        feat = np.ascontiguousarray(feat, np.float32)
        n_frames = feat.shape[1]
    tgt = None if target is None else np.ascontiguousarray(target, np.uint16)
    zc = np.zeros((S, T, N_CLASSES), np.float32) if logits else None
    zf = np.zeros((S, T, N_CLASSES), np.float32) if logits else None
    nl = np.zeros((S, T), np.float64) if nll else None
    m = _model(w)
    rc = L.orc_run(ctypes.byref(m), S, T, t0, _p(feat), n_frames, seed, _p(tgt), _p(h), _p(c), _p(f), _p(out),
                   _p(zc), _p(zf), _p(nl))
    if rc != 0:
        raise ValueError("oracle rejected the inputs")
    return dict(out=out, h=h, c=c, f=f, zc=zc, zf=zf, nll=nl)


def run_lanes(w: Weights, S: int, T: int, target, lanes, feat=None) -> dict:
    """Teacher-forced run of the subscale lanes [lanes[0], lanes[1]) only (they are
    independent given the target): dict(zc, zf [S][T][256], nll [S][T]) with the
    other lanes' entries zero."""
    B, H = w.B, w.H
    h = np.zeros((S * B, H), np.float32)
    c = np.full(S * B, 128, np.uint8)
    f = np.zeros(S * B, np.uint8)
    n_frames = 0
    if feat is not None:
        feat = np.ascontiguousarray(feat, np.float32)
        n_frames = feat.shape[1]
    tgt = np.ascontiguousarray(target, np.uint16)
    zc = np.zeros((S, T, N_CLASSES), np.float32)
    zf = np.zeros((S, T, N_CLASSES), np.float32)
    nl = np.zeros((S, T), np.float64)
    m = _model(w)
    rc = lib().orc_run_lanes(ctypes.byref(m), S, T, _p(feat), n_frames, _p(tgt), _p(h), _p(c), _p(f), _p(zc), _p(zf),
                             _p(nl), int(lanes[0]), int(lanes[1]))
    if rc != 0:
        raise ValueError("oracle rejected the inputs")
    return dict(zc=zc, zf=zf, nll=nl, h=h)


def fused_run(w: dict, S: int, N: int, feat=None, seed: int = 1, target=None, frame_len: int = 120) -> dict:
    """Fused Subscale WaveRNN 2x (Sec. 4.4): sample (target None) or teacher-force S
    utterances of N samples.  w: H, F and fp32 arrays R [3][H][H], I [3][H][6], b [3][H],
    O1 [4][Q][Q], b1 [4][Q], O2 [4][2][16][Q], b2 [4][2][16], optional Wc [3H][Dc].
    Returns dict(out [S][N] uint16, zc, zf [S][N][32], nll [S][N], h [S][H])."""
    H = int(w["H"])
    keep = {k: np.ascontiguousarray(w[k], np.float32) for k in ("R", "I", "b", "O1", "b1", "O2", "b2")}
    Wc = None if w.get("Wc") is None else np.ascontiguousarray(w["Wc"], np.float32)
    fp = lambda a: None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    m = _FusedModel(H, int(w["F"]), 0 if Wc is None else Wc.shape[1], frame_len,
                    fp(keep["R"]), fp(keep["I"]), fp(keep["b"]), fp(Wc), fp(keep["O1"]), fp(keep["b1"]),
                    fp(keep["O2"]), fp(keep["b2"]))
    n_frames = 0
    if feat is not None:
        feat = np.ascontiguousarray(feat, np.float32)
        n_frames = feat.shape[1]
    tgt = None if target is None else np.ascontiguousarray(target, np.uint16)
    out = np.zeros((S, N), np.uint16)
    zc = np.zeros((S, N, 32), np.float32)
    zf = np.zeros((S, N, 32), np.float32)
    nl = np.zeros((S, N), np.float64)
    h = np.zeros((S, H), np.float32)
    rc = lib().orc_fused_run(ctypes.byref(m), S, N, _p(feat), n_frames, seed, _p(tgt), _p(out), _p(zc), _p(zf),
                             _p(nl), _p(h))
    if rc != 0:
        raise ValueError("oracle rejected the inputs")
    return dict(out=out, zc=zc, zf=zf, nll=nl, h=h)


def ctx_cnn(w: dict, seq, s: int) -> np.ndarray:
    """Conditioning vectors [N/B][Dx] of sub-tensor s from the masked dilated CNN
    (Sec. 4.1, 5).  w: B, layers and fp32 arrays Win [Rc][2B], bin [Rc],
    Wc [layers][Cc][3][Rc], bc [layers][Cc], Wo [layers][Rc][Cc], bo [layers][Rc],
    Wp [Dx][Rc], bp [Dx]."""
    m = _cnn(w)
    B, Dx = m.B, m.Dx
    seq = np.ascontiguousarray(seq, np.uint16)
    out = np.zeros((len(seq) // B, Dx), np.float32)
    if lib().orc_ctx_cnn(ctypes.byref(m), _p(seq), len(seq), s, _p(out)) != 0:
        raise ValueError("oracle rejected the inputs")
    return out
