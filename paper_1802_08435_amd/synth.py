"""Seeded synthetic WaveRNN weights and inputs.

Holds none of the method's arithmetic: it only draws random arrays of the
shapes the model of Sec. 2 (Eq. 2) uses, for the GPU library, the oracle, the
tests and the benchmark alike.  There are no trained weights or speech data
here, so weights are ~N(0, 1/fan_in) and conditioning frames ~N(0, 1).
"""
from __future__ import annotations

import math

import numpy as np

N_CLASSES = 256
FRAME_LEN = 120          # 5 ms of 24 kHz audio per conditioning frame
COND_DIM = 64
CTX_DIM = 256            # subscale context: 128 preceding samples x (c, f)


def _normal(rng, shape, fan_in):
    return (rng.standard_normal(shape) / math.sqrt(fan_in)).astype(np.float32)


def make_weights(H: int, seed: int = 0, cond_dim: int = 0, B: int = 1, ctx_dim: int = 0,
                 block=None, density: float = 1.0, mask_seed: int = 3) -> dict:
    """Weights of one WaveRNN with H hidden units (H/2 coarse, H/2 fine).

    block = None (dense R) or (bh, bw) in {(4, 4), (16, 1)}: R keeps exactly
    round(density * n_blocks) random blocks per gate matrix (seeded by mask_seed),
    kept values ~N(0, 1/(density * H)); pruned entries are 0 and ``mask`` is the
    [3][H/bh][H/bw] uint8 block mask.  The masked entries of I (column 2 of the
    coarse rows) are filled with random values on purpose: the model ignores them."""
    assert H % 2 == 0
    Hh = H // 2
    rng = np.random.default_rng(seed)
    w = dict(H=H, B=B, frame_len=FRAME_LEN, block=block, mask=None)
    if block is None:
        w["R"] = _normal(rng, (3, H, H), H)
    else:
        bh, bw = block
        assert H % bh == 0 and H % bw == 0
        nbr, nbc = H // bh, H // bw
        mrng = np.random.default_rng(mask_seed)
        keep = int(round(density * nbr * nbc))
        mask = np.zeros((3, nbr * nbc), np.uint8)
        for g in range(3):
            mask[g, mrng.choice(nbr * nbc, keep, replace=False)] = 1
        mask = mask.reshape(3, nbr, nbc)
        vals = _normal(rng, (3, H, H), density * H)
        full = np.repeat(np.repeat(mask, bh, axis=1), bw, axis=2).astype(np.float32)
        w["R"] = (vals * full).astype(np.float32)
        w["mask"] = mask
    w["I"] = _normal(rng, (3, H, 3), 3)
    w["b"] = _normal(rng, (3, H), H)
    w["O1"] = _normal(rng, (Hh, Hh), Hh)
    w["b1"] = _normal(rng, (Hh,), Hh)
    w["O2"] = _normal(rng, (N_CLASSES, Hh), Hh)
    w["b2"] = _normal(rng, (N_CLASSES,), Hh)
    w["O3"] = _normal(rng, (Hh, Hh), Hh)
    w["b3"] = _normal(rng, (Hh,), Hh)
    w["O4"] = _normal(rng, (N_CLASSES, Hh), Hh)
    w["b4"] = _normal(rng, (N_CLASSES,), Hh)
    w["Wc"] = _normal(rng, (3 * H, cond_dim), cond_dim) if cond_dim else None
    w["Wx"] = _normal(rng, (3 * H, ctx_dim), ctx_dim) if ctx_dim else None
    return w


def make_fused_weights(H: int, F: int = 2, seed: int = 0, cond_dim: int = 0) -> dict:
    """Weights of a Fused Subscale WaveRNN 2x (Sec. 4.4) with H units (four
    quarters of Q = H/4), N(0, 1/fan_in): R [3][H][H], I [3][H][6] (last (c, f)
    of both sub-tensors, then their current coarse bytes), b [3][H], one MLP per
    (level, sub-tensor): O1 [4][Q][Q], b1 [4][Q], O2 [4][2][16][Q] (high and low
    nibble), b2 [4][2][16]; optional W_cond [3H][Dc].  The I columns a unit
    must ignore (the mask) hold random values on purpose."""
    assert H % 4 == 0
    Q = H // 4
    rng = np.random.default_rng(seed)
    w = dict(H=H, B=2, F=F, fused=True, frame_len=FRAME_LEN, block=None, mask=None)
    w["R"] = _normal(rng, (3, H, H), H)
    w["I"] = _normal(rng, (3, H, 6), 5)
    w["b"] = _normal(rng, (3, H), H)
    w["O1"] = _normal(rng, (4, Q, Q), Q)
    w["b1"] = _normal(rng, (4, Q), Q)
    w["O2"] = _normal(rng, (4, 2, 16, Q), Q)
    w["b2"] = _normal(rng, (4, 2, 16), Q)
    w["Wc"] = _normal(rng, (3 * H, cond_dim), cond_dim) if cond_dim else None
    w["Wx"] = None
    return w


def make_cnn_weights(B: int, Rc: int = 768, Cc: int = 384, Dx: int = 256, layers: int = 10, seed: int = 5) -> dict:
    """The masked dilated CNN that conditions a Subscale WaveRNN (Sec. 4.1, 5):
    Win [Rc][2B], per layer Wc [Cc][3][Rc] (taps k, k + d, k + 2d), Wo [Rc][Cc],
    and Wp [Dx][Rc], N(0, 1/fan_in), biases N(0, 0.1^2); the paper's widths by
    default (768 residual, 384 convolution channels, ten layers).  The residual
    stream grows over the layers (to about 4 at ten), so Wp is scaled by 1/4:
    context values of order one."""
    rng = np.random.default_rng(seed)
    b = lambda *shape: (0.1 * rng.standard_normal(shape)).astype(np.float32)
    return dict(B=B, layers=layers, Win=_normal(rng, (Rc, 2 * B), 2 * B), bin=b(Rc),
                Wc=_normal(rng, (layers, Cc, 3, Rc), 3 * Rc), bc=b(layers, Cc),
                Wo=_normal(rng, (layers, Rc, Cc), Cc), bo=b(layers, Rc),
                Wp=_normal(rng, (Dx, Rc), 16 * Rc), bp=b(Dx))


def features(S: int, T: int, cond_dim: int = COND_DIM, seed: int = 2, frame_len: int = FRAME_LEN,
             per_stream_seed: bool = False) -> np.ndarray:
    """Conditioning frames [S][ceil(T/frame_len)][cond_dim] ~N(0, 1)."""
    n_frames = max(1, -(-T // frame_len))
    if per_stream_seed:
        return np.stack([np.random.default_rng(seed + s).standard_normal((n_frames, cond_dim))
                         for s in range(S)]).astype(np.float32)
    rng = np.random.default_rng(seed)
    return rng.standard_normal((S, n_frames, cond_dim)).astype(np.float32)


def target_signal(S: int, T: int, seed: int = 4, kind: str = "sines") -> np.ndarray:
    """16-bit offset-binary sample sequences [S][T] (coarse byte = high 8 bits).

    kind='sines': three sinusoids summing to -10 dBFS plus N(0, 1e-3) noise;
    kind='uniform': uniform random 16-bit words."""
    rng = np.random.default_rng(seed)
    if kind == "uniform":
        return rng.integers(0, 65536, size=(S, T), dtype=np.uint16)
    t = np.arange(T) / 24000.0
    out = np.empty((S, T), np.uint16)
    amp = 10 ** (-10 / 20) / 3
    for s in range(S):
        f = rng.uniform(80, 4000, size=3)
        ph = rng.uniform(0, 2 * np.pi, size=3)
        x = sum(amp * np.sin(2 * np.pi * f[k] * t + ph[k]) for k in range(3))
        x = x + rng.normal(0, 1e-3, size=T)
        q = np.clip(np.round(x * 32767), -32768, 32767).astype(np.int64) + 32768
        out[s] = q.astype(np.uint16)
    return out


PRESETS = {
    # name: (H, cond_dim, B, ctx_dim, block, bf16, streams, samples)
    "tiny": (64, 0, 1, 0, None, False, 1, 2400),
    "dense896": (896, COND_DIM, 1, 0, None, True, 1, 24000),
    "sparse2048_4x4": (2048, COND_DIM, 1, 0, (4, 4), True, 1, 24000),
    "sparse2048_16x1": (2048, COND_DIM, 1, 0, (16, 1), True, 1, 24000),
    "subscale16": (896, COND_DIM, 16, CTX_DIM, None, True, 1, 24000),
    "multi64": (896, COND_DIM, 1, 0, None, True, 64, 48000),
    "multi4": (896, COND_DIM, 1, 0, None, True, 4, 24000),   # Sec. 2.1's batch-4 point
    "subscale16_h4": (896, COND_DIM, 16, CTX_DIM, None, True, 1, 24000),
    "subscale16_h4a1": (896, COND_DIM, 16, CTX_DIM, None, True, 1, 24000),
    "subscale16_cnn": (896, COND_DIM, 16, CTX_DIM, None, True, 1, 24000),
}
# Subscale presets in the paper's order with a future horizon (Sec. 4.2):
# lane s starts F + 1 + A steps after lane s - 1 (24,000 samples with F = 4:
# 1,500 + 15 x (5 + A) steps), A the steps by which its context is formed
# ahead; the others run lockstep rows.
HORIZON = {"subscale16_h4": 4, "subscale16_h4a1": 4, "subscale16_cnn": 223}
LEAD = {"subscale16_h4a1": 1}   # the lead is switched off at create (E_UNSUPPORTED) for now
# Subscale conditioned by the masked dilated CNN at the paper's widths (Sec. 4.1, 5): it
# reaches 124 rows ahead, so with F = 223 it runs ahead in chunks of 100 rows (Sec. 4.2's L).
CNN = {"subscale16_cnn": dict(Rc=768, Cc=384, layers=10)}


# Fused Subscale WaveRNN 2x (Sec. 4.4): WaveRNN-896 with its state in quarters,
# F = 2 as the paper uses, 24,000 samples (12,000 positions per sub-tensor).
FUSED = {"fused896": (896, 2, COND_DIM, 1, 24000)}


def preset(name: str, seed: int = 0) -> dict:
    if name in FUSED:
        H, F, Dc, S, T = FUSED[name]
        w = make_fused_weights(H, F=F, seed=seed, cond_dim=Dc)
        w.update(name=name, bf16=True, streams=S, samples=T)
        return w
    H, Dc, B, Dx, block, bf16, S, T = PRESETS[name]
    w = make_weights(H, seed=seed, cond_dim=Dc, B=B, ctx_dim=Dx, block=block,
                     density=0.04 if block else 1.0)
    w.update(name=name, bf16=bf16, streams=S, samples=T)
    if name in HORIZON:
        w["F"] = HORIZON[name]
        w["A"] = LEAD.get(name, 0)
    if name in CNN:
        w["cnn"] = make_cnn_weights(B, Dx=Dx, **CNN[name])
    return w
