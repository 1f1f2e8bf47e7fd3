"""The draw's edge cases on every kernel path, through the C ABI.

A model whose weights are all zero except the two output biases keeps h = 0,
so its logits are exactly those biases (Eq. 2 with relu(0) = 0): the coarse
bias is +100 on the four classes 37..40 and -200 elsewhere (logits far above
exp's range, so the max shift matters, and 252 zero-probability classes), the
fine bias +50 on the sixteen classes 240..255 and -200 elsewhere.  The
inverse-CDF draw then has a closed form: c = 37 + floor(4 U_c), f = 240 +
floor(16 U_f), exactly (the running sums are small integers), for the oracle
and for every kernel.  The uniforms include the most extreme ones of the
first 2^22 steps of the stream (reached through t0 on the batch-1 paths).
"""
import functools
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from oracle import oracle as O  # noqa: E402
from paper_1802_08435_amd import synth, wavernn  # noqa: E402


def host(t):
    return t.cpu().numpy()


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def edge_model(H, B=1, Dx=0, block=None):
    w = synth.make_weights(H, seed=3, cond_dim=0, B=B, ctx_dim=Dx, block=block, density=0.25 if block else 1.0)
    for k in ("R", "I", "b", "O1", "b1", "O2", "O3", "b3", "O4") + (("Wx",) if Dx else ()):
        w[k] = np.zeros_like(w[k])
    w["b2"] = np.full(256, -200.0, np.float32)
    w["b2"][37:41] = 100.0
    w["b4"] = np.full(256, -200.0, np.float32)
    w["b4"][240:256] = 50.0
    return w


def expected(seed, stream, t0, n):
    """The closed-form samples of steps t0 .. t0+n-1 from the oracle's (numpy-pinned) uniforms."""
    out = []
    for t in range(t0, t0 + n):
        uc, uf = O.uniforms(seed, stream, t)
        out.append(256 * (37 + math.floor(4 * uc)) + 240 + math.floor(16 * uf))
    return np.array(out, np.uint16)


@functools.lru_cache(maxsize=None)
def extreme_steps(seed, stream, n=1 << 22):
    """Steps of the smallest and largest coarse and fine uniforms among the first n (numpy's Philox)."""
    from numpy.random import Philox
    v = (0 + (stream << 64) - 1) % 2**256
    ctr = np.array([(v >> (64 * k)) & (2**64 - 1) for k in range(4)], dtype=np.uint64)
    raw = Philox(key=seed, counter=ctr).random_raw(4 * n).reshape(n, 4)
    u = (raw[:, :2] >> np.uint64(40)).astype(np.int64)
    steps = sorted({int(u[:, 0].argmin()), int(u[:, 0].argmax()), int(u[:, 1].argmin()), int(u[:, 1].argmax())})
    return steps, u.min(axis=0), u.max(axis=0)


@pytest.mark.parametrize("kind", ["single-workgroup", "persistent", "block-sparse", "concurrent", "batched-2",
                                  "batched-8"])
def test_edge_draws_at_extreme_uniforms(kind):
    """Batch-1 style paths: windows of 48 steps around the most extreme
    uniforms of the first 2^22 steps of each stream, entered through t0."""
    H, S, dtype, block, ms = {"single-workgroup": (64, 1, "f32", None, 1), "persistent": (256, 1, "bf16", None, 1),
                              "block-sparse": (256, 1, "bf16", (4, 4), 1), "concurrent": (256, 3, "bf16", None, 3),
                              "batched-2": (256, 6, "bf16", None, 6), "batched-8": (256, 40, "bf16", None, 40)}[kind]
    w = edge_model(H, block=block)
    m = wavernn.Model(w, dtype=dtype, r_format="bsr4x4" if block else "dense", max_streams=ms)
    assert m.path(S)[0] == ("batched" if kind.startswith("batched") else kind)
    seed = 7
    streams = sorted({0, S - 1, S // 2})
    for st in streams:
        steps, lo, hi = extreme_steps(seed, st)
        assert lo.max() < 64 and hi.min() > 2**24 - 64      # within 2^-18 of both ends of [0, 1)
        for t_ex in steps:
            t0 = max(0, t_ex - 24)
            print(f"edges {kind} stream {st} t0 {t0}", flush=True)
            init = m.new_state(S)
            init["t0"] = t0
            out = host(m.sample(48, seed=seed, n_streams=S, init=init))
            m.device_status()
            np.testing.assert_array_equal(out[st], expected(seed, st, t0, 48), err_msg=f"{kind} stream {st} t0 {t0}")
    m.close()


@pytest.mark.parametrize("F", [-1, 2])
def test_edge_draws_subscale(F):
    """Subscale lanes (B = 16, lockstep and future horizon 2): every sample of
    1,600 (100 rows) has the closed form of its lane's Philox stream."""
    B = 16
    w = edge_model(256, B=B, Dx=64)
    w["F"] = F
    m = wavernn.Model(w)
    N = B * 100
    out = host(m.sample(N, seed=9))[0]
    m.device_status()
    for s in range(B):
        np.testing.assert_array_equal(out[s::B], expected(9, s, 0, N // B), err_msg=f"lane {s}")
    m.close()
