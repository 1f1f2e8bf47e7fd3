"""Python binding of libwavernn (``include/wavernn.h``): argument marshalling only.

Every step of sampling runs in the HIP kernels of ``libwavernn.so``; PyTorch only
supplies device memory and the current HIP stream.  There is no fallback: if the
library is not built, every entry point raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwavernn.so")
_lib = None

OK, E_INVALID, E_UNSUPPORTED, E_OOM, E_HIP, E_DEVICE = range(6)
F32, BF16 = 0, 1
R_DENSE, R_BSR_4X4, R_BSR_16X1 = 0, 1, 2
PATHS = {0: "single-workgroup", 1: "persistent", 2: "batched", 3: "block-sparse", 4: "concurrent", 5: "fused"}


class WaveRNNError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"wavernn status {status}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("hidden", "cond_dim", "frame_len", "subscale", "ctx_dim",
                                               "weight_dtype", "r_format", "max_streams", "future_horizon",
                                               "context_lead", "fused")]


_FP = ctypes.POINTER(ctypes.c_float)


class CtxCnn(ctypes.Structure):
    _fields_ = [("res_channels", ctypes.c_int32), ("conv_channels", ctypes.c_int32), ("layers", ctypes.c_int32)] + [
        (n, _FP) for n in ("Win", "bin", "Wc", "bc", "Wo", "bo", "Wp", "bp")]


class Weights(ctypes.Structure):
    _fields_ = [("R", _FP), ("R_block_mask", ctypes.POINTER(ctypes.c_uint8)), ("I", _FP), ("b", _FP),
                ("W_cond", _FP), ("W_ctx", _FP)] + [(n, _FP) for n in ("O1", "b1", "O2", "b2", "O3", "b3", "O4", "b4")] + [
        ("ctx_cnn", ctypes.POINTER(CtxCnn))]


class State(ctypes.Structure):
    _fields_ = [("h", ctypes.c_void_p), ("c_prev", ctypes.c_void_p), ("f_prev", ctypes.c_void_p),
                ("t0", ctypes.c_int64)]


def lib():
    """Load libwavernn.so (built by ``__graft_entry__.build()``); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
        L.wavernn_create.restype = ctypes.c_int
        L.wavernn_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Weights), ctypes.POINTER(vp)]
        L.wavernn_destroy.restype = None
        L.wavernn_destroy.argtypes = [vp]
        L.wavernn_sample.restype = ctypes.c_int
        L.wavernn_sample.argtypes = [vp, i32, i64, vp, i64, u64, ctypes.POINTER(State), vp, ctypes.POINTER(State), vp]
        L.wavernn_sample_noalloc.restype = ctypes.c_int
        L.wavernn_sample_noalloc.argtypes = [vp, i32, i64, vp, i64, u64, ctypes.POINTER(State), vp,
                                             ctypes.POINTER(State), vp]
        L.wavernn_sample_steps.restype = ctypes.c_int
        L.wavernn_sample_steps.argtypes = [vp, i32, i64, vp, i64, u64, i64, i64, ctypes.POINTER(State), vp,
                                           ctypes.POINTER(State), vp]
        L.wavernn_schedule_steps.restype = i64
        L.wavernn_schedule_steps.argtypes = [vp, i64]
        L.wavernn_score_teacher_forced.restype = ctypes.c_int
        L.wavernn_score_teacher_forced.argtypes = [vp, i32, i64, vp, i64, vp, ctypes.POINTER(State), vp, vp, vp, vp]
        L.wavernn_device_status.restype = ctypes.c_int
        L.wavernn_device_status.argtypes = [vp, vp]
        L.wavernn_debug_uniforms.restype = ctypes.c_int
        L.wavernn_debug_uniforms.argtypes = [u64, u64, i64, i64, vp, vp]
        L.wavernn_set_trace.restype = ctypes.c_int
        L.wavernn_set_trace.argtypes = [vp, vp, i64]
        L.wavernn_debug_sync_floor.restype = ctypes.c_int
        L.wavernn_debug_sync_floor.argtypes = [vp, i64, ctypes.POINTER(ctypes.c_double), vp]
        L.wavernn_tune.restype = ctypes.c_int
        L.wavernn_tune.argtypes = [vp, i64, i32, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(i32), vp]
        L.wavernn_set_placement.restype = ctypes.c_int
        L.wavernn_set_placement.argtypes = [vp, i32]
        L.wavernn_model_path.restype = i32
        L.wavernn_model_path.argtypes = [vp, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.wavernn_ctx_cnn_run.restype = ctypes.c_int
        L.wavernn_ctx_cnn_run.argtypes = [vp, i32, i64, vp, vp, vp]
        L.wavernn_last_error.restype = ctypes.c_char_p
        L.wavernn_last_error.argtypes = []
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise WaveRNNError(status, lib().wavernn_last_error().decode())


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _f32(a):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=np.float32)


class Model:
    """A WaveRNN on the current GPU.

    ``w`` is a dict of fp32 arrays (keys of ``include/wavernn.h``'s weights:
    R, I, b, O1, b1, O2, b2, O3, b3, O4, b4, optional Wc, Wx, mask) plus H,
    frame_len, B and, for subscale, F (future horizon; -1 or absent: lockstep rows) and A (steps by which
    the context is formed ahead, with F only; absent: 0).  dtype 'bf16' or 'f32' is the weight storage; r_format is
    'dense', 'bsr4x4' or 'bsr16x1'.  A Fused Subscale 2x model (``fused`` true) has B = 2, F, I [3][H][6],
    O1 [4][Q][Q], b1 [4][Q], O2 [4][2][16][Q], b2 [4][2][16] and no O3, b3, O4, b4.  A subscale model
    with a future horizon may carry ``cnn``: the conditioning CNN's arrays (Win, bin, Wc, bc, Wo, bo,
    Wp, bp; include/wavernn.h's wavernn_ctx_cnn), which replaces the window context."""

    def __init__(self, w: dict, dtype: str = "bf16", r_format: str = "dense", max_streams: int = 1):
        L = lib()
        self.H = int(w["H"])
        Wc, Wx = _f32(w.get("Wc")), _f32(w.get("Wx"))
        self.cond_dim = 0 if Wc is None else Wc.shape[1]
        self.frame_len = int(w.get("frame_len", 120))
        self.B = int(w.get("B", 1))
        self.F = int(w.get("F", -1))
        self.A = int(w.get("A", 0))
        self.fused = bool(w.get("fused", False))
        cfg = Config(self.H, self.cond_dim, self.frame_len, self.B, 0 if Wx is None else Wx.shape[1],
                     {"bf16": BF16, "f32": F32}[dtype],
                     {"dense": R_DENSE, "bsr4x4": R_BSR_4X4, "bsr16x1": R_BSR_16X1}[r_format], max_streams,
                     self.F, self.A, int(self.fused))
        keep = {k: _f32(w.get(k)) for k in ("R", "I", "b", "O1", "b1", "O2", "b2", "O3", "b3", "O4", "b4")}
        mask = None if w.get("mask") is None else np.ascontiguousarray(w["mask"], dtype=np.uint8)
        fp = lambda a: None if a is None else a.ctypes.data_as(_FP)
        ws = Weights(fp(keep["R"]), None if mask is None else mask.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                     fp(keep["I"]), fp(keep["b"]), fp(Wc), fp(Wx),
                     *[fp(keep[k]) for k in ("O1", "b1", "O2", "b2", "O3", "b3", "O4", "b4")])
        self.cnn = w.get("cnn")
        if self.cnn is not None:
            ck = {k: _f32(self.cnn[k]) for k in ("Win", "bin", "Wc", "bc", "Wo", "bo", "Wp", "bp")}
            cc = CtxCnn(ck["Win"].shape[0], ck["bc"].shape[1] if int(self.cnn["layers"]) > 0 else 128,
                        int(self.cnn["layers"]), *[fp(ck[k]) for k in ("Win", "bin", "Wc", "bc", "Wo", "bo", "Wp", "bp")])
            ws.ctx_cnn = ctypes.pointer(cc)
            keep["_cnn"] = (ck, cc)
        h = ctypes.c_void_p()
        _check(L.wavernn_create(ctypes.byref(cfg), ctypes.byref(ws), ctypes.byref(h)))
        self._h = h
        self.max_streams = max_streams

    def close(self):
        if getattr(self, "_h", None):
            lib().wavernn_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def path(self, n_streams: int = 1):
        """(kernel name, grid, block) serving a call on n_streams streams."""
        g, b = ctypes.c_int32(), ctypes.c_int32()
        p = lib().wavernn_model_path(self._h, n_streams, ctypes.byref(g), ctypes.byref(b))
        return PATHS.get(p, str(p)), g.value, b.value

    @staticmethod
    def _state(st):
        if st is None:
            return None
        return State(st["h"].data_ptr(), st["c"].data_ptr(), st["f"].data_ptr(), int(st.get("t0", 0)))

    def new_state(self, n_streams: int = 1):
        """Default state: h [S B][H] (fused: [S][H]), last bytes [S B] (fused: [2 S])."""
        import torch
        d = torch.device("cuda")
        nh = n_streams if self.fused else n_streams * self.B
        return dict(h=torch.zeros(nh, self.H, device=d),
                    c=torch.full((n_streams * self.B,), 128, dtype=torch.uint8, device=d),
                    f=torch.zeros(n_streams * self.B, dtype=torch.uint8, device=d), t0=0)

    def sample(self, n_samples: int, cond=None, seed: int = 1, n_streams: int = 1, init=None, final=None,
               out=None, stream=None, noalloc: bool = False):
        """Draw n_samples per utterance; returns the [n_streams][n_samples] uint16 tensor.
        ``final`` (a dict from new_state) receives the state after the last sample.
        ``noalloc``: call wavernn_sample_noalloc (the library's per-device workspace,
        no device allocation; ``out`` must then be given)."""
        import torch
        if out is None:
            if noalloc:
                raise ValueError("sample(noalloc=True) needs a preallocated out tensor")
            out = torch.empty(n_streams, n_samples, dtype=torch.uint16, device="cuda")
        n_frames = 0 if cond is None else cond.shape[1]
        si, sf = self._state(init), self._state(final)
        fn = lib().wavernn_sample_noalloc if noalloc else lib().wavernn_sample
        _check(fn(self._h, n_streams, n_samples, _ptr(cond), n_frames, seed,
                  None if si is None else ctypes.byref(si), _ptr(out),
                  None if sf is None else ctypes.byref(sf), _stream(stream)))
        if final is not None:
            final["t0"] = (init["t0"] if init is not None else 0) + n_samples
        return out

    def schedule_steps(self, n_samples: int) -> int:
        """Steps of the schedule of a subscale call of n_samples per utterance (-1: not served)."""
        return int(lib().wavernn_schedule_steps(self._h, n_samples))

    def sample_steps(self, out, step0: int, n_steps: int, cond=None, seed: int = 1, init=None, final=None,
                     stream=None):
        """Run steps [step0, step0 + n_steps) of the schedule of a subscale call
        whose whole utterances are out [S][n_samples] (uint16, holding every
        sample earlier steps made); init: the state after step0 - 1 (a dict from
        new_state, required when step0 > 0); final receives the state after the
        last step (include/wavernn.h, wavernn_sample_steps)."""
        S, n_samples = out.shape
        n_frames = 0 if cond is None else cond.shape[1]
        si, sf = self._state(init), self._state(final)
        _check(lib().wavernn_sample_steps(self._h, S, n_samples, _ptr(cond), n_frames, seed, step0, n_steps,
                                          None if si is None else ctypes.byref(si), _ptr(out),
                                          None if sf is None else ctypes.byref(sf), _stream(stream)))
        return out

    def score(self, target, cond=None, init=None, logits: bool = True, nll: bool = True, stream=None):
        """Teacher-forced logits [S][T][256] x2 (fused: [S][T][32]) and NLL [S][T] (nats) on target [S][T] uint16."""
        import torch
        S, T = target.shape
        nz = 32 if self.fused else 256
        zc = torch.empty(S, T, nz, device="cuda") if logits else None
        zf = torch.empty(S, T, nz, device="cuda") if logits else None
        nl = torch.empty(S, T, device="cuda") if nll else None
        n_frames = 0 if cond is None else cond.shape[1]
        si = self._state(init)
        _check(lib().wavernn_score_teacher_forced(self._h, S, T, _ptr(cond), n_frames, _ptr(target),
                                                  None if si is None else ctypes.byref(si),
                                                  _ptr(zc), _ptr(zf), _ptr(nl), _stream(stream)))
        return dict(zc=zc, zf=zf, nll=nl)

    def ctx_cnn(self, seq, stream=None):
        """Conditioning CNN over whole utterances seq [S][N] uint16: tensor [S][B][N/B][Dx]."""
        import torch
        S, N = seq.shape
        out = torch.empty(S, self.B, N // self.B, int(self.cnn["Wp"].shape[0]), device="cuda")
        _check(lib().wavernn_ctx_cnn_run(self._h, S, N, _ptr(seq), _ptr(out), _stream(stream)))
        return out

    def set_trace(self, buf=None):
        """Record per-phase timestamps of later persistent-kernel calls into buf,
        an int64 cuda tensor [steps][32] (None: stop)."""
        n = 0 if buf is None else buf.shape[0]
        _check(lib().wavernn_set_trace(self._h, _ptr(buf), n))
        self._trace = buf

    def device_status(self, stream=None):
        _check(lib().wavernn_device_status(self._h, _stream(stream)))

    def tune(self, n_steps: int = 2048, rounds: int = 2, stream=None) -> dict:
        """Time each placement of the persistent kernel's workgroups over the
        XCDs and keep the fastest (include/wavernn.h, wavernn_tune): returns
        {"chosen": candidate or -1, "us_per_step": [64] floats, -1 = does not fit}."""
        us = (ctypes.c_float * 64)()
        ch = ctypes.c_int32()
        _check(lib().wavernn_tune(self._h, n_steps, rounds, us, ctypes.byref(ch), _stream(stream)))
        return {"chosen": ch.value, "us_per_step": [float(x) for x in us]}

    def set_placement(self, candidate: int):
        """Candidate placement as in tune(); -1: the default."""
        _check(lib().wavernn_set_placement(self._h, candidate))

    def sync_floor(self, n_steps: int = 20000, stream=None) -> float:
        """Microseconds per step of the persistent kernel's exchange pattern alone
        (same grid and exchanged words, no arithmetic); waits for it."""
        us = ctypes.c_double()
        _check(lib().wavernn_debug_sync_floor(self._h, n_steps, ctypes.byref(us), _stream(stream)))
        return us.value


def debug_uniforms(seed: int, stream_id: int, t0: int, n: int):
    """(coarse, fine) uniforms the kernels draw for steps t0..t0+n-1: tensor [n][2]."""
    import torch
    out = torch.empty(n, 2, device="cuda")
    _check(lib().wavernn_debug_uniforms(seed, stream_id, t0, n, _ptr(out), _stream()))
    return out
