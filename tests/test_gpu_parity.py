"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Bars: free-running fp32 samples of the single-workgroup kernel are bit-identical
to the oracle's for the same Philox uniforms (the kernel follows the oracle's
evaluation order); teacher-forced logits of the persistent bf16-weight kernel
are within 2e-2 absolute of the oracle run on the same bf16-rounded weights
(the kernel sums in another order); its free-running draws are checked for
validity against the oracle's logits on the same trajectory.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from oracle import oracle as O  # noqa: E402
from paper_1802_08435_amd import synth, wavernn  # noqa: E402

BF16_TOL = 2e-2
# The context lead (A > 0) is switched off at create: a traced launch with a
# lead of 1 had a bounded wait expire and the cause is not found.
LEAD_OFF = pytest.mark.skip(reason="context lead switched off: a traced launch with A = 1 had a bounded wait "
                                   "expire, cause not found")


def cuda(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.cpu().numpy()


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def test_uniforms_match_oracle():
    for seed, stream, t0 in [(1, 0, 0), (7, 3, 123456), (2**63 + 5, 63, 2**33)]:
        g = host(wavernn.debug_uniforms(seed, stream, t0, 300))
        for i in range(0, 300, 7):
            assert tuple(g[i]) == O.uniforms(seed, stream, t0 + i)


# ------------------------------------------------------------------ small kernel

def test_tiny_free_running_bit_identical():
    w = synth.preset("tiny")
    m = wavernn.Model(w, dtype="f32")
    assert m.path()[0] == "single-workgroup"
    fin = m.new_state()
    out = host(m.sample(2400, seed=1, final=fin))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w), 1, 2400, seed=1)
    np.testing.assert_array_equal(out, ref["out"])
    np.testing.assert_array_equal(host(fin["h"]), ref["h"])
    assert int(host(fin["c"])[0]) == int(ref["c"][0]) and int(host(fin["f"])[0]) == int(ref["f"][0])


@pytest.mark.parametrize("kind", ["sines", "uniform"])
def test_tiny_teacher_forced_logits_exact(kind):
    w = synth.preset("tiny")
    tgt = synth.target_signal(2, 2400, kind=kind)
    m2 = wavernn.Model(w, dtype="f32", max_streams=2)
    r = m2.score(cuda(tgt))
    m2.device_status()
    ref = O.run(O.Weights.from_dict(w), 2, 2400, target=tgt, logits=True, nll=True)
    np.testing.assert_array_equal(host(r["zc"]), ref["zc"])
    np.testing.assert_array_equal(host(r["zf"]), ref["zf"])
    np.testing.assert_allclose(host(r["nll"]), ref["nll"], rtol=1e-5, atol=1e-5)


def test_tiny_bf16_weights_bit_identical_and_multistream_chunked():
    w = synth.make_weights(64, seed=5, cond_dim=8)
    feat = synth.features(3, 1000, cond_dim=8)
    m = wavernn.Model(w, dtype="bf16", max_streams=3)
    s1 = m.new_state(3)
    a = host(m.sample(600, cond=cuda(feat), seed=11, n_streams=3, final=s1))
    b = host(m.sample(400, cond=cuda(feat), seed=11, n_streams=3, init=s1, final=s1))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), 3, 1000, feat=feat, seed=11)
    np.testing.assert_array_equal(np.concatenate([a, b], axis=1), ref["out"])
    np.testing.assert_array_equal(host(s1["h"]), ref["h"])


# ------------------------------------------------------------- persistent kernel

def _tf_compare(w, T, S=1, cond_dim=0, seed_t=4):
    feat = synth.features(S, T, cond_dim=cond_dim) if cond_dim else None
    tgt = np.concatenate([synth.target_signal(1, T, seed=seed_t), synth.target_signal(1, T, seed=seed_t, kind="uniform")])[:S]
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    r = m.score(cuda(tgt), cond=None if feat is None else cuda(feat))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=tgt, logits=True, nll=True)
    return m, {k: host(v) for k, v in r.items()}, ref


def _targets(S, T, seed=4):
    """Sine and uniform-byte targets, alternating over the streams."""
    kinds = ["sines", "uniform"]
    return np.concatenate([synth.target_signal(1, T, seed=seed + s, kind=kinds[s % 2]) for s in range(S)])


@pytest.mark.parametrize("H", [128, 256, 384])
def test_persistent_teacher_forced_small_sizes(H):
    w = synth.make_weights(H, seed=1, cond_dim=16)
    m, r, ref = _tf_compare(w, 300, S=1, cond_dim=16)
    assert m.path()[0] == "persistent"
    dc = np.abs(r["zc"] - ref["zc"]).max()
    df = np.abs(r["zf"] - ref["zf"]).max()
    assert dc <= 1e-3 and df <= 1e-3, (dc, df)
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-4, atol=1e-3)


@pytest.mark.parametrize("H,S", [(128, 6), (256, 9), (384, 16), (256, 24), (256, 40)])
def test_batched_teacher_forced_small_sizes(H, S):
    """Several utterances in one launch (groups of 2 vectors up to 16
    utterances, 4 up to 32, 8 above; S=9 leaves an idle vector in the last
    group; up to 4 utterances take the concurrent path instead): logits of
    every stream against the oracle."""
    w = synth.make_weights(H, seed=1, cond_dim=16)
    T = 200
    feat = synth.features(S, T, cond_dim=16, per_stream_seed=True)
    tgt = _targets(S, T)
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    assert m.path(S)[0] == "batched"
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=tgt, logits=True, nll=True)
    dc = np.abs(r["zc"] - ref["zc"]).max()
    df = np.abs(r["zf"] - ref["zf"]).max()
    assert dc <= 1e-3 and df <= 1e-3, (dc, df)
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-4, atol=1e-3)


@pytest.mark.parametrize("S,T", [(12, 240), (33, 120)])
def test_batched_dense896_teacher_forced_within_bf16_tolerance(S, T):
    """WaveRNN-896 with groups of 2 vectors (12 utterances) and of 8 (33: heads
    evaluate their own slice of units and exchange y; one live vector in the
    last group)."""
    w = synth.preset("dense896")
    feat = synth.features(S, T, per_stream_seed=True)
    tgt = _targets(S, T)
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    assert m.path(S)[0] == "batched"
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=tgt, logits=True, nll=True)
    d = max(np.abs(r["zc"] - ref["zc"]).max(), np.abs(r["zf"] - ref["zf"]).max())
    assert d <= BF16_TOL, d
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-3, atol=2e-2)


def test_dense896_teacher_forced_within_bf16_tolerance():
    w = synth.preset("dense896")
    m, r, ref = _tf_compare(w, 960, S=1, cond_dim=64)
    assert m.path()[0] == "persistent"
    d = max(np.abs(r["zc"] - ref["zc"]).max(), np.abs(r["zf"] - ref["zf"]).max())
    assert d <= BF16_TOL, d
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-3, atol=2e-2)


def _check_draws_valid(z, u, k, delta):
    """k was drawn from softmax(z) with uniform u by inverse CDF, up to a shift of
    the class boundaries by at most delta (probability mass)."""
    z = z.astype(np.float64)
    k = k.astype(np.int64)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    C = np.cumsum(p, axis=1)
    lo = np.where(k > 0, C[np.arange(len(k)), np.maximum(k - 1, 0)], 0.0)
    hi = C[np.arange(len(k)), k]
    return (u >= lo - delta) & (u <= hi + delta)


def test_dense896_free_running_draws_are_valid():
    """Sample 2400 steps on the GPU, teacher-force the oracle on that trajectory
    and check every GPU draw against the oracle's distribution and uniforms."""
    w = synth.preset("dense896")
    T = 2400
    feat = synth.features(1, T)
    m = wavernn.Model(w, dtype="bf16")
    out = host(m.sample(T, cond=cuda(feat), seed=1))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), 1, T, feat=feat, target=out, logits=True)
    u = np.array([O.uniforms(1, 0, t) for t in range(T)])
    c, f = out[0] >> 8, out[0] & 255
    okc = _check_draws_valid(ref["zc"][0], u[:, 0], c, 1e-3)
    okf = _check_draws_valid(ref["zf"][0], u[:, 1], f, 1e-3)
    assert okc.all() and okf.all(), (np.flatnonzero(~okc)[:10], np.flatnonzero(~okf)[:10])
    # not a degenerate trajectory
    assert len(np.unique(out)) > 100


@pytest.mark.parametrize("S", [9, 40])
def test_batched_free_running_draws_valid_and_chunked_equals_one_call(S):
    """9 or 40 utterances in one launch: every draw is valid under the oracle's
    logits on the GPU trajectory and the stream's own Philox uniforms, and two
    chained calls give the same samples and state as one."""
    w = synth.make_weights(256, seed=3, cond_dim=8)
    T = 500
    feat = synth.features(S, T, cond_dim=8, per_stream_seed=True)
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    fin = m.new_state(S)
    whole = host(m.sample(T, cond=cuda(feat), seed=7, n_streams=S, final=fin))
    st = m.new_state(S)
    a = host(m.sample(300, cond=cuda(feat), seed=7, n_streams=S, final=st))
    b = host(m.sample(200, cond=cuda(feat), seed=7, n_streams=S, init=st, final=st))
    m.device_status()
    np.testing.assert_array_equal(np.concatenate([a, b], axis=1), whole)
    np.testing.assert_array_equal(host(st["h"]), host(fin["h"]))
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=whole, logits=True)
    for s_ in range(S):
        u = np.array([O.uniforms(7, s_, t) for t in range(T)])
        c, f = whole[s_] >> 8, whole[s_] & 255
        okc = _check_draws_valid(ref["zc"][s_], u[:, 0], c, 1e-3)
        okf = _check_draws_valid(ref["zf"][s_], u[:, 1], f, 1e-3)
        assert okc.all() and okf.all(), (s_, np.flatnonzero(~okc)[:10], np.flatnonzero(~okf)[:10])
    assert len({tuple(x[:50]) for x in whole}) == S     # streams differ


# ------------------------------------------------------------- concurrent batch-1 launches

@pytest.mark.parametrize("H,S", [(256, 3), (896, 4)])
def test_concurrent_streams_teacher_forced_free_running_and_chunked(H, S):
    """2 to 4 utterances of a dense model run as concurrent batch-1 launches
    (one grid per utterance on internal streams): teacher-forced logits
    against the oracle, free-running draws valid on each utterance's Philox
    stream, two chained calls equal one, and the caller's stream sees every
    result (stream-ordered)."""
    w = synth.preset("dense896") if H == 896 else synth.make_weights(H, seed=5, cond_dim=16)
    Dc = w["Wc"].shape[1]
    T = 240
    feat = synth.features(S, T, cond_dim=Dc, per_stream_seed=True)
    tgt = _targets(S, T)
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    assert m.path(S)[0] == "concurrent"
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    W = O.Weights.from_dict(w, bf16=True)
    ref = O.run(W, S, T, feat=feat, target=tgt, logits=True, nll=True)
    d = max(np.abs(r["zc"] - ref["zc"]).max(), np.abs(r["zf"] - ref["zf"]).max())
    assert d <= BF16_TOL, d
    fin = m.new_state(S)
    whole = host(m.sample(T, cond=cuda(feat), seed=9, n_streams=S, final=fin))
    st = m.new_state(S)
    a = host(m.sample(100, cond=cuda(feat), seed=9, n_streams=S, final=st))
    b = host(m.sample(T - 100, cond=cuda(feat), seed=9, n_streams=S, init=st, final=st))
    m.device_status()
    np.testing.assert_array_equal(np.concatenate([a, b], axis=1), whole)
    np.testing.assert_array_equal(host(st["h"]), host(fin["h"]))
    ref = O.run(W, S, T, feat=feat, target=whole, logits=True)
    for s_ in range(S):
        u = np.array([O.uniforms(9, s_, t) for t in range(T)])
        okc = _check_draws_valid(ref["zc"][s_], u[:, 0], whole[s_] >> 8, 1e-3)
        okf = _check_draws_valid(ref["zf"][s_], u[:, 1], whole[s_] & 255, 1e-3)
        assert okc.all() and okf.all(), (s_, np.flatnonzero(~okc)[:10], np.flatnonzero(~okf)[:10])
    assert len({tuple(x[:50]) for x in whole}) == S


# ------------------------------------------------------------- subscale

@pytest.mark.parametrize("H,B,S", [(256, 8, 2), (128, 16, 1), (128, 16, 3), (128, 16, 4)])   # 4 x 16: 64 vectors, the most
def test_subscale_teacher_forced_small_sizes(H, B, S):
    """Subscale (Sec. 4): B lanes per utterance in lockstep, each conditioned on
    the 128 samples before its own (same-row samples masked); 3 utterances of
    16 lanes make groups of 8 vectors."""
    w = synth.make_weights(H, seed=6, cond_dim=16, B=B, ctx_dim=256)
    T = 40 * B
    feat = synth.features(S, T, cond_dim=16, per_stream_seed=True)
    tgt = _targets(S, T)
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    assert m.path(S)[0] == "batched"
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=tgt, logits=True, nll=True)
    dc = np.abs(r["zc"] - ref["zc"]).max()
    df = np.abs(r["zf"] - ref["zf"]).max()
    assert dc <= 1e-3 and df <= 1e-3, (dc, df)
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-4, atol=1e-3)


def test_subscale16_dense896_teacher_forced_within_bf16_tolerance():
    w = synth.preset("subscale16")
    T = 960
    feat = synth.features(1, T)
    tgt = _targets(1, T)
    m = wavernn.Model(w, dtype="bf16")
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), 1, T, feat=feat, target=tgt, logits=True, nll=True)
    d = max(np.abs(r["zc"] - ref["zc"]).max(), np.abs(r["zf"] - ref["zf"]).max())
    assert d <= BF16_TOL, d
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-3, atol=2e-2)


@pytest.mark.parametrize("H,B,S,F,A", [(256, 8, 2, 1, 0), (128, 16, 1, 2, 0), (256, 4, 2, 0, 0),
                                       (128, 16, 3, 1, 0), (128, 16, 4, 2, 0),
                                       pytest.param(256, 8, 2, 1, 1, marks=LEAD_OFF),
                                       pytest.param(128, 16, 1, 2, 2, marks=LEAD_OFF),
                                       pytest.param(256, 4, 2, 0, 3, marks=LEAD_OFF),
                                       pytest.param(128, 16, 3, 1, 1, marks=LEAD_OFF)])
def test_subscale_horizon_teacher_forced_small_sizes(H, B, S, F, A):
    """Subscale in the paper's order with future horizon F (Sec. 4.2): lane s
    runs position i at step i + s (F + 1 + A) and its context holds samples
    of earlier sub-tensors up to position i + F, formed A steps ahead (3
    utterances of 16 lanes make groups of 8 vectors).  Logits of every
    sample against the oracle, which generates sub-tensor by sub-tensor and
    knows no A: the schedule must not change what is computed."""
    w = synth.make_weights(H, seed=6, cond_dim=16, B=B, ctx_dim=256)
    w["F"], w["A"] = F, A
    T = 40 * B
    feat = synth.features(S, T, cond_dim=16, per_stream_seed=True)
    tgt = _targets(S, T)
    m = wavernn.Model(w, dtype="bf16", max_streams=S)
    assert m.path(S)[0] == "batched"
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=tgt, logits=True, nll=True)
    dc = np.abs(r["zc"] - ref["zc"]).max()
    df = np.abs(r["zf"] - ref["zf"]).max()
    assert dc <= 1e-3 and df <= 1e-3, (dc, df)
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-4, atol=1e-3)


@pytest.mark.parametrize("name", ["subscale16_h4", pytest.param("subscale16_h4a1", marks=LEAD_OFF)])
def test_subscale16_horizon_dense896_teacher_forced_within_bf16_tolerance(name):
    w = synth.preset(name)
    T = 960
    feat = synth.features(1, T)
    tgt = _targets(1, T)
    m = wavernn.Model(w, dtype="bf16")
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), 1, T, feat=feat, target=tgt, logits=True, nll=True)
    d = max(np.abs(r["zc"] - ref["zc"]).max(), np.abs(r["zf"] - ref["zf"]).max())
    assert d <= BF16_TOL, d
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-3, atol=2e-2)


@pytest.mark.parametrize("A", [0, pytest.param(1, marks=LEAD_OFF)])
def test_subscale_horizon_free_running_draws_valid_and_final_state(A):
    """Free-running with horizon F = 2 (context formed A steps ahead): every
    lane's draw is valid under the oracle's logits on the GPU trajectory with
    the lane's Philox stream indexed by position, and the final state is each
    lane's after its last position."""
    B, T, F = 8, 480, 2
    w = synth.make_weights(256, seed=7, cond_dim=16, B=B, ctx_dim=256)
    w["F"], w["A"] = F, A
    feat = synth.features(1, T, cond_dim=16)
    m = wavernn.Model(w, dtype="bf16")
    fin = m.new_state()
    out = host(m.sample(T, cond=cuda(feat), seed=3, final=fin))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), 1, T, feat=feat, target=out, logits=True)
    u = np.array([O.uniforms(3, n % B, n // B) for n in range(T)])
    c, f = out[0] >> 8, out[0] & 255
    okc = _check_draws_valid(ref["zc"][0], u[:, 0], c, 1e-3)
    okf = _check_draws_valid(ref["zf"][0], u[:, 1], f, 1e-3)
    assert okc.all() and okf.all(), (np.flatnonzero(~okc)[:10], np.flatnonzero(~okf)[:10])
    assert len(np.unique(out)) > 50
    last = out[0, T - B:]                            # the last sample of lane s is T - B + s
    np.testing.assert_array_equal(host(fin["c"]), last >> 8)
    np.testing.assert_array_equal(host(fin["f"]), last & 255)
    np.testing.assert_allclose(host(fin["h"]), ref["h"], atol=1e-2)


def test_subscale_free_running_draws_are_valid():
    """Every lane's draw is valid under the oracle's logits on the GPU
    trajectory, with the lane's Philox stream indexed by row."""
    B, T = 8, 480
    w = synth.make_weights(256, seed=7, cond_dim=16, B=B, ctx_dim=256)
    feat = synth.features(1, T, cond_dim=16)
    m = wavernn.Model(w, dtype="bf16")
    out = host(m.sample(T, cond=cuda(feat), seed=3))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), 1, T, feat=feat, target=out, logits=True)
    u = np.array([O.uniforms(3, n % B, n // B) for n in range(T)])
    c, f = out[0] >> 8, out[0] & 255
    okc = _check_draws_valid(ref["zc"][0], u[:, 0], c, 1e-3)
    okf = _check_draws_valid(ref["zf"][0], u[:, 1], f, 1e-3)
    assert okc.all() and okf.all(), (np.flatnonzero(~okc)[:10], np.flatnonzero(~okf)[:10])
    assert len(np.unique(out)) > 50


def test_persistent_chunked_equals_one_call():
    w = synth.make_weights(256, seed=2, cond_dim=8)
    feat = synth.features(1, 900, cond_dim=8)
    m = wavernn.Model(w, dtype="bf16")
    whole = host(m.sample(900, cond=cuda(feat), seed=5))
    st = m.new_state()
    a = host(m.sample(500, cond=cuda(feat), seed=5, final=st))
    b = host(m.sample(400, cond=cuda(feat), seed=5, init=st, final=st))
    m.device_status()
    np.testing.assert_array_equal(np.concatenate([a, b], axis=1), whole)


def test_invalid_calls_return_errors_without_launching():
    w = synth.preset("tiny")
    m = wavernn.Model(w, dtype="f32")
    out = torch.empty(2, 10, dtype=torch.uint16, device="cuda")
    with pytest.raises(wavernn.WaveRNNError) as e:
        m.sample(10, n_streams=2, out=out)
    assert e.value.status == wavernn.E_INVALID
    wc = synth.make_weights(64, cond_dim=4)
    mc = wavernn.Model(wc, dtype="f32")
    with pytest.raises(wavernn.WaveRNNError):
        mc.sample(10)                      # conditioning missing
    with pytest.raises(wavernn.WaveRNNError):
        mc.sample(500, cond=cuda(synth.features(1, 100, cond_dim=4)))   # too few frames
    assert host(m.sample(0)).shape == (1, 0)


_EDGE_KINDS = {"single-workgroup": dict(H=64), "persistent": dict(H=256), "block-sparse": dict(H=256, block=(4, 4), density=0.1),
               "batched": dict(H=256, S=5), "subscale": dict(H=256, B=4), "subscale-horizon": dict(H=256, B=4, F=1)}


def test_lead_is_switched_off():
    w = synth.preset("subscale16_h4a1")
    with pytest.raises(wavernn.WaveRNNError) as err:
        wavernn.Model(w)
    assert err.value.status == wavernn.E_UNSUPPORTED and "switched off" in str(err.value)


@pytest.mark.parametrize("kind", sorted(_EDGE_KINDS))
def test_degenerate_calls_on_every_path(kind):
    """Zero-length calls succeed, launch nothing and leave outputs and the
    final state untouched; a subscale length that is not a multiple of B and
    more utterances than the model was created for are rejected."""
    e = dict(_EDGE_KINDS[kind])
    H, S, B = e.pop("H"), e.pop("S", 1), e.pop("B", 1)
    kw = dict(cond_dim=16)
    if "block" in e:
        kw.update(block=e.pop("block"), density=e.pop("density"))
    if B > 1:
        kw.update(B=B, ctx_dim=256)
    w = synth.make_weights(H, seed=13, **kw)
    w.update({k: v for k, v in e.items()})
    m = wavernn.Model(w, dtype="f32" if kind == "single-workgroup" else "bf16", r_format="bsr4x4" if "block" in kw else "dense",
                      max_streams=S)
    assert m.path(S)[0] == {"subscale-horizon": "batched", "subscale": "batched"}.get(kind, kind)
    feat = cuda(synth.features(S, 8 * B, cond_dim=16, per_stream_seed=True))
    out = torch.full((S, 0), 7, dtype=torch.uint16, device="cuda")
    fin = m.new_state(S)
    fin["h"].fill_(0.25)
    m.sample(0, cond=feat, n_streams=S, out=out, final=fin)
    r = m.score(torch.empty(S, 0, dtype=torch.uint16, device="cuda"), cond=feat)
    m.device_status()
    assert host(r["zc"]).shape == (S, 0, 256) and host(r["nll"]).shape == (S, 0)
    assert (host(fin["h"]) == 0.25).all() and (host(fin["c"]) == 128).all()
    if B > 1:
        with pytest.raises(wavernn.WaveRNNError) as err:
            m.sample(B + 1, cond=feat, n_streams=S)
        assert err.value.status == wavernn.E_INVALID
    with pytest.raises(wavernn.WaveRNNError) as err:
        m.sample(B, cond=cuda(synth.features(S + 1, 8 * B, cond_dim=16)), n_streams=S + 1)
    assert err.value.status == wavernn.E_INVALID
    # the model still samples after the rejected calls
    o = host(m.sample(2 * B, cond=feat, n_streams=S, seed=4))
    m.device_status()
    assert o.shape == (S, 2 * B)


# ------------------------------------------------------------- block-sparse R

_FMT = {(4, 4): "bsr4x4", (16, 1): "bsr16x1"}


@pytest.mark.parametrize("H,block,density", [(128, (4, 4), 0.25), (256, (16, 1), 0.1), (256, (4, 4), 0.04)])
def test_block_sparse_teacher_forced_small_sizes(H, block, density):
    """Sparse WaveRNN (Sec. 3.2): R kept in 4x4 or 16x1 blocks; the oracle runs
    the dense R with the pruned blocks zero."""
    w = synth.make_weights(H, seed=8, cond_dim=16, block=block, density=density)
    m, r, ref = _tf_compare_fmt(w, 300, _FMT[block], cond_dim=16)
    assert m.path()[0] == "block-sparse"
    dc = np.abs(r["zc"] - ref["zc"]).max()
    df = np.abs(r["zf"] - ref["zf"]).max()
    assert dc <= 1e-3 and df <= 1e-3, (dc, df)
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-4, atol=1e-3)


def _tf_compare_fmt(w, T, fmt, S=1, cond_dim=0):
    feat = synth.features(S, T, cond_dim=cond_dim, per_stream_seed=True) if cond_dim else None
    tgt = _targets(S, T)
    m = wavernn.Model(w, dtype="bf16", r_format=fmt, max_streams=S)
    r = m.score(cuda(tgt), cond=None if feat is None else cuda(feat))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=tgt, logits=True, nll=True)
    return m, {k: host(v) for k, v in r.items()}, ref


def test_block_sparse_all_blocks_kept_matches_dense_kernel():
    """With every block kept the block-sparse kernel computes the dense model:
    its logits agree with the dense persistent kernel's and the oracle's."""
    w = synth.make_weights(256, seed=9, cond_dim=16, block=(4, 4), density=1.0)
    assert w["mask"].all()
    T = 240
    m, r, ref = _tf_compare_fmt(w, T, "bsr4x4", cond_dim=16)
    assert m.path()[0] == "block-sparse"
    feat = synth.features(1, T, cond_dim=16, per_stream_seed=True)
    md = wavernn.Model(w, dtype="bf16")
    assert md.path()[0] == "persistent"
    rd = {k: host(v) for k, v in md.score(cuda(_targets(1, T)), cond=cuda(feat)).items()}
    md.device_status()
    for k in ("zc", "zf"):
        assert np.abs(r[k] - ref[k]).max() <= 1e-3
        assert np.abs(r[k] - rd[k]).max() <= 1e-3


@pytest.mark.parametrize("name,T", [("sparse2048_4x4", 240), ("sparse2048_16x1", 120)])
def test_sparse2048_teacher_forced_within_bf16_tolerance(name, T):
    w = synth.preset(name)
    m, r, ref = _tf_compare_fmt(w, T, _FMT[w["block"]], cond_dim=64)
    assert m.path()[0] == "block-sparse"
    d = max(np.abs(r["zc"] - ref["zc"]).max(), np.abs(r["zf"] - ref["zf"]).max())
    assert d <= BF16_TOL, d
    np.testing.assert_allclose(r["nll"], ref["nll"], rtol=1e-3, atol=2e-2)


def test_sparse2048_free_running_draws_are_valid():
    w = synth.preset("sparse2048_4x4")
    T = 480
    feat = synth.features(1, T)
    m = wavernn.Model(w, dtype="bf16", r_format="bsr4x4")
    out = host(m.sample(T, cond=cuda(feat), seed=1))
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), 1, T, feat=feat, target=out, logits=True)
    u = np.array([O.uniforms(1, 0, t) for t in range(T)])
    c, f = out[0] >> 8, out[0] & 255
    okc = _check_draws_valid(ref["zc"][0], u[:, 0], c, 1e-3)
    okf = _check_draws_valid(ref["zf"][0], u[:, 1], f, 1e-3)
    assert okc.all() and okf.all(), (np.flatnonzero(~okc)[:10], np.flatnonzero(~okf)[:10])
    assert len(np.unique(out)) > 50


def test_block_sparse_streams_and_chunks():
    """Two utterances (one launch each) sampled in two chained calls equal one
    call, and the final state matches."""
    w = synth.make_weights(256, seed=10, cond_dim=8, block=(16, 1), density=0.1)
    S, T = 2, 500
    feat = synth.features(S, T, cond_dim=8, per_stream_seed=True)
    m = wavernn.Model(w, dtype="bf16", r_format="bsr16x1", max_streams=S)
    assert m.path(S)[0] == "block-sparse"
    fin = m.new_state(S)
    whole = host(m.sample(T, cond=cuda(feat), seed=4, n_streams=S, final=fin))
    st = m.new_state(S)
    a = host(m.sample(320, cond=cuda(feat), seed=4, n_streams=S, final=st))
    b = host(m.sample(180, cond=cuda(feat), seed=4, n_streams=S, init=st, final=st))
    m.device_status()
    np.testing.assert_array_equal(np.concatenate([a, b], axis=1), whole)
    np.testing.assert_array_equal(host(st["h"]), host(fin["h"]))
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, T, feat=feat, target=whole, logits=True)
    for s_ in range(S):
        u = np.array([O.uniforms(4, s_, t) for t in range(T)])
        okc = _check_draws_valid(ref["zc"][s_], u[:, 0], whole[s_] >> 8, 1e-3)
        okf = _check_draws_valid(ref["zf"][s_], u[:, 1], whole[s_] & 255, 1e-3)
        assert okc.all() and okf.all()


@pytest.mark.parametrize("name", ["dense896", "sparse2048_4x4", "multi64", "subscale16", "subscale16_h4"])
def test_sync_floor_runs_below_the_step_time(name):
    """The exchange-only kernel (same grid, same words per step; for the
    batched launches the batched kernel with its arithmetic compiled out)
    completes and costs less per step than the sampling kernel it mirrors."""
    w = synth.preset(name)
    S, B = w["streams"], w["B"]
    m = wavernn.Model(w, dtype="bf16", r_format=_FMT.get(w["block"], "dense"), max_streams=S)
    rows = 3000 // B * 10 if B > 1 else 3000
    floor = m.sync_floor(rows)
    T = B * rows
    feat = cuda(synth.features(S, T, per_stream_seed=S > 1))
    steps = rows + ((B - 1) * (w["F"] + 1) if w.get("F", -1) >= 0 else 0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    m.sample(T, cond=feat, seed=1, n_streams=S)
    e1.record()
    torch.cuda.synchronize()
    m.device_status()
    step = e0.elapsed_time(e1) * 1000.0 / steps
    assert 0.5 < floor < step, (floor, step)


@pytest.mark.parametrize("kind", ["persistent", "block-sparse", "batched", "concurrent", "subscale",
                                  "subscale-horizon"])
@pytest.mark.parametrize("T", [1, 2, 65])
def test_short_runs_match_the_oracle(kind, T):
    """Edge lengths: one step (no unit iteration at all), two steps, and one
    step past a 64-step uniform batch, on every multi-workgroup path."""
    H, S, fmt, B = 256, 1, "dense", 1
    kw = dict(cond_dim=16)
    if kind == "block-sparse":
        kw.update(block=(4, 4), density=0.1)
        fmt = "bsr4x4"
    if kind == "batched":
        S = 5
    if kind == "concurrent":
        S = 2
    if kind.startswith("subscale"):
        B = 4
        kw.update(B=B, ctx_dim=256)
    w = synth.make_weights(H, seed=12, **kw)
    if kind == "subscale-horizon":
        w["F"] = 1
    n = T * B
    feat = synth.features(S, n, cond_dim=16, per_stream_seed=True)
    tgt = _targets(S, n)
    m = wavernn.Model(w, dtype="bf16", r_format=fmt, max_streams=S)
    assert m.path(S)[0] == {"subscale": "batched", "subscale-horizon": "batched"}.get(kind, kind)
    r = {k: host(v) for k, v in m.score(cuda(tgt), cond=cuda(feat)).items()}
    m.device_status()
    ref = O.run(O.Weights.from_dict(w, bf16=True), S, n, feat=feat, target=tgt, logits=True, nll=True)
    assert np.abs(r["zc"] - ref["zc"]).max() <= 1e-3 and np.abs(r["zf"] - ref["zf"]).max() <= 1e-3
    out = host(m.sample(n, cond=cuda(feat), seed=3, n_streams=S))
    m.device_status()
    assert out.shape == (S, n)
