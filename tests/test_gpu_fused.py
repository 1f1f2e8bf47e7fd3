"""GPU parity of the Fused Subscale WaveRNN 2x kernel (Sec. 4.4) against the
oracle's orc_fused_run, through the C ABI.

Bars: teacher-forced nibble logits within 1e-3 at small sizes and 2e-2 (bf16
weights, another summation order) at H = 896, NLL alike; free-running draws
valid under the oracle's logits on the GPU's own trajectory with the oracle's
Philox words; point-mass heads give exactly the oracle's samples.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from oracle import oracle as O  # noqa: E402
from paper_1802_08435_amd import synth, wavernn  # noqa: E402

BF16_TOL = 2e-2
KEYS = ("R", "I", "b", "O1", "b1", "O2", "b2", "Wc")


def cuda(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.cpu().numpy()


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def oracle_weights(w):
    """The weights as the library stores them (bf16, round to nearest even)."""
    d = {k: (None if w.get(k) is None else O.bf16_round(w[k])) for k in KEYS}
    d.update(H=w["H"], F=w["F"])
    return d


def words(seed, stream, i):
    """The four uniforms of Philox counter (i, stream): coarse high, coarse low, fine high, fine low nibble."""
    return [int(x >> np.uint64(40)) / 2.0**24 for x in O.philox4x64_10([i, stream, 0, 0], [seed, 0])]


def targets(S, N, seed=4):
    kinds = ["sines", "uniform"]
    return np.concatenate([synth.target_signal(1, N, seed=seed + s, kind=kinds[s % 2]) for s in range(S)])


def score_both(w, S, N, cond_dim, seed_t=4):
    feat = synth.features(S, N, cond_dim=cond_dim, per_stream_seed=True) if cond_dim else None
    tgt = targets(S, N, seed_t)
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    assert m.path(S)[0] == "fused"
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=None if feat is None else cuda(feat)).items()}
    m.device_status()
    ref = O.fused_run(oracle_weights(w), S, N, feat=feat, target=tgt, frame_len=w["frame_len"])
    return m, r, ref


@pytest.mark.parametrize("H,F,S", [(128, 0, 1), (128, 2, 2), (256, 2, 1), (256, 5, 2), (384, 1, 1)])
def test_fused_teacher_forced_small_sizes(H, F, S):
    """Several tiles and heads, both sub-tensors' ramps (sub-tensor 1 idle for
    the first F + 1 steps, sub-tensor 0 for the last), 2 utterances."""
    w = synth.make_fused_weights(H, F=F, seed=1, cond_dim=16)
    print(f"fused tf H={H} F={F} S={S}", flush=True)
    m, r, ref = score_both(w, S, 2 * 150, 16)
    dc = np.abs(r["zc"] - ref["zc"]).max()
    df = np.abs(r["zf"] - ref["zf"]).max()
    assert dc <= 1e-3 and df <= 1e-3, (dc, df)
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-4, atol=2e-3)
    m.close()


def test_fused896_teacher_forced_within_bf16_tolerance():
    w = synth.preset("fused896")
    m, r, ref = score_both(w, 1, 960, 64)
    d = max(np.abs(r["zc"] - ref["zc"]).max(), np.abs(r["zf"] - ref["zf"]).max())
    assert d <= BF16_TOL, d
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-3, atol=4e-2)
    m.close()


def _check_nibbles_valid(z16, u, k, delta=1e-3):
    """k drawn from softmax(z16) with uniform u by inverse CDF, class boundaries shifted by at most delta."""
    z = z16.astype(np.float64)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    C = np.cumsum(p, axis=1)
    idx = np.arange(len(k))
    lo = np.where(k > 0, C[idx, np.maximum(k - 1, 0)], 0.0)
    hi = C[idx, k]
    return (u >= lo - delta) & (u <= hi + delta)


def _validate_trajectory(w, out, feat, seed, S, n_check=None):
    """Teacher-force the oracle on the GPU's samples; every nibble the GPU drew
    among the first n_check samples (all by default) must be the inverse-CDF
    class of the oracle's softmax at the Philox word of its position and
    sub-tensor.  A prefix of n_check samples is replayed with 2 (F + 1) samples
    more, so that sub-tensor 0 is still active wherever sub-tensor 1's checked
    positions see it (Sec. 4.2 horizon)."""
    N = out.shape[1] if n_check is None else min(out.shape[1], n_check + 2 * (w["F"] + 1))
    out = out[:, :N]
    ref = O.fused_run(oracle_weights(w), S, N, feat=feat, target=out, frame_len=w["frame_len"])
    if n_check is not None:
        N = n_check
        out = out[:, :N]
        ref = {k: v[:, :N] for k, v in ref.items() if k != "h"}
    for u_ in range(S):
        U = np.array([words(seed, 2 * u_ + (n % 2), n // 2) for n in range(N)])
        c, f = out[u_].astype(np.int64) >> 8, out[u_].astype(np.int64) & 255
        parts = [(ref["zc"][u_][:, :16], U[:, 0], c >> 4), (ref["zc"][u_][:, 16:], U[:, 1], c & 15),
                 (ref["zf"][u_][:, :16], U[:, 2], f >> 4), (ref["zf"][u_][:, 16:], U[:, 3], f & 15)]
        for z, uu, k in parts:
            ok = _check_nibbles_valid(z, uu, k)
            assert ok.all(), (u_, np.flatnonzero(~ok)[:10])
    return ref


def test_fused896_free_running_draws_valid_and_final_state():
    w = synth.preset("fused896")
    S, N = 2, 2400
    feat = synth.features(S, N, per_stream_seed=True)
    m = wavernn.Model(w, max_streams=S)
    fin = m.new_state(S)
    out = host(m.sample(N, cond=cuda(feat), seed=7, n_streams=S, final=fin))
    m.device_status()
    ref = _validate_trajectory(w, out, feat, 7, S)
    assert all(len(np.unique(out[u_])) > 200 for u_ in range(S))
    # last samples of both sub-tensors; the state after the whole call
    c, f = host(fin["c"]), host(fin["f"])
    for u_ in range(S):
        assert (c[2 * u_], f[2 * u_]) == (out[u_, -2] >> 8, out[u_, -2] & 255)
        assert (c[2 * u_ + 1], f[2 * u_ + 1]) == (out[u_, -1] >> 8, out[u_, -1] & 255)
    assert np.abs(host(fin["h"]) - ref["h"]).max() <= 2e-2
    m.close()


def _point_mass_model(H=128, F=2):
    """Zero weights except the nibble biases: the state stays 0, so every
    nibble's logits are its bias row.  Head k puts +100 on high nibble 1 + k
    (max shift: logits far above exp's range), -200 elsewhere except a block of
    four equal low nibbles (zero-probability classes around them)."""
    w = synth.make_fused_weights(H, F=F, seed=0, cond_dim=0)
    for k in ("R", "I", "b", "O1", "b1", "O2"):
        w[k] = np.zeros_like(w[k])
    b2 = np.full((4, 2, 16), -200.0, np.float32)
    for k in range(4):
        b2[k, 0, 1 + k] = 100.0
        b2[k, 1, 4 * k:4 * k + 4] = 0.0
    w["b2"] = b2
    return w


def test_fused_point_mass_and_zero_probability_nibbles():
    """Edge cases of the 16-way draws: a point mass with logits near +100, and
    zero-probability classes (-200) around a block of four equal ones, over
    3,200 uniforms that come within 1e-3 of both ends of [0, 1): high nibbles
    are the point masses, low nibbles the oracle's draw bit for bit (equal
    weights: floor(4 U) into the block), never a zero-probability class."""
    w = _point_mass_model()
    S, N = 2, 2 * 400
    m = wavernn.Model(w, max_streams=S)
    out = host(m.sample(N, seed=3, n_streams=S))
    m.device_status()
    ref = O.fused_run(oracle_weights(w), S, N, seed=3, frame_len=w["frame_len"])
    np.testing.assert_array_equal(out, ref["out"])
    allu = np.array([words(3, st, i) for st in range(2 * S) for i in range(N // 2)])
    assert allu.min() < 1e-3 and allu.max() > 1 - 1e-3
    for u_ in range(S):
        for n in range(N):
            s = n % 2
            c, f = int(out[u_, n]) >> 8, int(out[u_, n]) & 255
            assert (c >> 4, f >> 4) == (1 + s, 3 + s)
            assert c & 15 in range(4 * s, 4 * s + 4) and f & 15 in range(4 * (2 + s), 4 * (2 + s) + 4)
            U = words(3, 2 * u_ + s, n // 2)
            assert c & 15 == 4 * s + math.floor(4 * U[1]) and f & 15 == 4 * (2 + s) + math.floor(4 * U[3])
    # NLL of a point-mass target: four nibbles, each log(1 + 3 e^-300) + log 4 or ~0
    tgt = out.copy()
    r = m.score(cuda(tgt))
    m.device_status()
    np.testing.assert_allclose(host(r["nll"]), 2 * math.log(4.0), rtol=0, atol=1e-4)
    m.close()


def test_fused_degenerate_calls():
    w = synth.make_fused_weights(128, F=2, seed=2, cond_dim=0)
    m = wavernn.Model(w)
    out = torch.zeros(1, 8, dtype=torch.uint16, device="cuda")
    m.sample(0, out=out)                                  # nothing launched
    with pytest.raises(wavernn.WaveRNNError):
        m.sample(7, out=out)                              # odd length
    st = m.new_state()
    st["t0"] = 2
    with pytest.raises(wavernn.WaveRNNError):
        m.sample(8, out=out, init=st)                     # no resume inside the fused schedule
    # one position per sub-tensor: F + 2 steps, sub-tensor 1 alone at the last
    one = host(m.sample(2, seed=5, out=out[:, :2]))
    m.device_status()
    ref = O.fused_run(oracle_weights(w), 1, 2, seed=5, target=one, frame_len=w["frame_len"])
    U = [words(5, s, 0) for s in range(2)]
    for s in range(2):
        c, f = int(one[0, s]) >> 8, int(one[0, s]) & 255
        for z, uu, k in ((ref["zc"][0][s, :16], U[s][0], c >> 4), (ref["zc"][0][s, 16:], U[s][1], c & 15),
                         (ref["zf"][0][s, :16], U[s][2], f >> 4), (ref["zf"][0][s, 16:], U[s][3], f & 15)):
            assert _check_nibbles_valid(z[None, :], np.array([uu]), np.array([k])).all()
    m.close()


def test_fused896_full_length_call():
    """The benchmarked call (24,000 samples, one launch of 12,003 steps): the
    first 2,400 samples are valid draws under the oracle, and the whole call
    is a plausible trajectory (both sub-tensors active to the end, state
    bounded, last samples handed over)."""
    w = synth.preset("fused896")
    N = w["samples"]
    feat = synth.features(1, N)
    m = wavernn.Model(w)
    fin = m.new_state()
    out = host(m.sample(N, cond=cuda(feat), seed=1, final=fin))
    m.device_status()
    _validate_trajectory(w, out, feat, 1, 1, n_check=2400)
    for s in range(2):
        tail = out[0, N - 2000 + s::2]
        assert len(np.unique(tail)) > 100
    h = host(fin["h"])
    assert np.isfinite(h).all() and np.abs(h).max() <= 1.0
    assert host(fin["c"])[1] == out[0, -1] >> 8 and host(fin["f"])[0] == out[0, -2] & 255
    m.close()
