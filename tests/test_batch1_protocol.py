"""A CPU model of the batch-1 persistent kernel's exchange protocol with
mirrors (CPU only; the kernel is in wr_persist.hip and wr_unit.h).

Heads, mirrors and units run the kernel's order of publishes and waits, one
read of one word per scheduling step, under random interleavings with
strongly skewed speeds.  A workgroup is one agent; where two of its waves wait
for different words at the same time (the draw wave and the gate threads),
the model reads the two sets in a random interleaving.  Words carry the
kernel's tags:

* single-buffered words (y slices, coarse partial logits, the units'
  coarse-column words, the mirrors' words) hold the parity of step + 1;
* double-buffered words (the units' fine-row words and the fine partial
  logits) of step s sit in buffer s mod 2 and hold the parity of s / 2 + 1.
* the leads' XCD words are written once, at the start.

A reader accepts a word whose bit matches, and the model then checks that the
word was written for the awaited step: a match on another step is a misread.

What the model leaves out: values, barriers inside a workgroup, memory
ordering of the hardware (every write is visible to the next read) and the
bounded waits' clock.
"""
import random

import pytest


def run(NH=3, NU=4, T=14, seed=0, pf_double=True, gf_double=True, heads_check_first=True, max_ticks=2_000_000):
    rng = random.Random(seed)
    NM = NH
    mem = {}

    def single(name, i, s):
        return (name, i), (s + 1) & 1

    def double(name, i, s, on):
        if not on:
            return single(name, i, s)
        return (name, i, s & 1), ((s >> 1) + 1) & 1

    def pub(key_bit, s):
        key, bit = key_bit
        return ("w", key, bit, s)

    def wait(key_bit, s):
        key, bit = key_bit
        return ("r", key, bit, s)

    def mixed(a, b):
        """Two waves' reads, in a random interleaving."""
        a, b = list(a), list(b)
        while a or b:
            if a and (not b or rng.random() < 0.5):
                yield a.pop(0)
            else:
                yield b.pop(0)

    PC = lambda j, s: single("PC", j, s)
    PF = lambda j, s: double("PF", j, s, pf_double)
    GA = lambda k, s: single("GA", k, s)
    GF = lambda k, s: double("GF", k, s, gf_double)
    HF = lambda m, s: single("HF", m, s)
    YC = lambda j, s: single("YC", j, s)
    YF = lambda j, s: single("YF", j, s)

    def coarse_words(s):
        return [wait(GA(k, s), s) for k in range(NU)] + [wait(HF(m, s), s) for m in range(NM)]

    # The XCD check at the start: every lead (head or mirror) publishes its
    # XCD word once and reads every lead's before it uses local stores.
    XC = lambda i: (("XC", i), 1)

    def xcd_check(i):
        yield pub(XC(i), 0)
        for ii in range(NH + NM):
            yield wait(XC(ii), 0)

    def head(j):
        if heads_check_first:           # the kernel's order: before step 0's coarse gates
            yield from xcd_check(j)
        yield from coarse_words(0)
        if not heads_check_first:
            yield from xcd_check(j)
        for s in range(T):
            yield pub(YC(j, s), s)
            yield pub(PC(j, s), s)
            # the draw wave gathers the coarse partials, the gate threads the fine words
            yield from mixed([wait(PC(jj, s), s) for jj in range(NH)], [wait(GF(k, s), s) for k in range(NU)])
            yield pub(YF(j, s), s)
            yield pub(PF(j, s), s)
            # the draw wave gathers the fine partials, the gate threads the next coarse words
            nxt = coarse_words(s + 1) if s + 1 < T else []
            yield from mixed([wait(PF(jj, s), s) for jj in range(NH)], nxt)

    def mirror(m):
        yield from xcd_check(NH + m)    # before the words of step 0
        yield pub(HF(m, 0), 0)
        for s in range(T):
            yield from mixed([wait(PC(jj, s), s) for jj in range(NH)], [wait(GF(k, s), s) for k in range(NU)])
            if s + 1 < T:
                yield pub(HF(m, s + 1), s + 1)
            yield from (wait(PF(jj, s), s) for jj in range(NH))

    def unit(k):
        yield pub(GA(k, 0), 0)
        yield pub(GF(k, 0), 0)
        for t in range(T - 1):
            for j in range(NH):
                yield wait(YC(j, t), t)
            yield pub(GA(k, t + 1), t + 1)
            for j in range(NH):
                yield wait(YF(j, t), t)
            yield pub(GF(k, t + 1), t + 1)

    agents = [head(j) for j in range(NH)] + [mirror(m) for m in range(NM)] + [unit(k) for k in range(NU)]
    speed = [rng.random() ** 4 + 0.002 for _ in agents]     # some agents hundreds of times slower
    cur = [next(a) for a in agents]
    live = set(range(len(agents)))

    def ready(i):
        kind, key, bit, _ = cur[i]
        return kind == "w" or mem.get(key, (0, -1))[0] == bit

    for _ in range(max_ticks):
        if not live:
            return None
        rd = [i for i in live if ready(i)]
        if not rd:
            return f"deadlock (a word lost or never written): {[cur[i] for i in sorted(live)][:4]}"
        i = rng.choices(rd, weights=[speed[x] for x in rd])[0]
        kind, key, bit, s = cur[i]
        if kind == "w":
            mem[key] = (bit, s)
        elif mem[key][1] != s:
            return f"misread: {key} awaited for step {s}, holds step {mem[key][1]}"
        try:
            cur[i] = next(agents[i])
        except StopIteration:
            live.discard(i)
    return "ran out of ticks"


@pytest.mark.parametrize("NH,NU", [(2, 3), (3, 4), (4, 2)])
def test_mirrored_protocol_has_no_lost_or_misread_word(NH, NU):
    """Random interleavings, skewed speeds: every awaited word is read with the
    step it was awaited for, and nothing waits forever."""
    fails = [(sd, e) for sd in range(40) for e in [run(NH=NH, NU=NU, seed=sd)] if e]
    assert not fails, fails[:2]


def test_the_model_catches_single_buffered_fine_words():
    """The model is not blind: with the fine partial logits or the fine rows'
    words in one buffer, some interleaving misreads a word (a mirror reads the
    fine partials of a step after publishing its words for the next one, and
    the units publish fine words a mirror may not have read yet)."""
    assert any(run(seed=sd, pf_double=False) for sd in range(200))
    assert any(run(seed=sd, gf_double=False) for sd in range(200))


def test_the_xcd_check_comes_before_any_wait_on_another_lead():
    """The leads' XCD check (every head and mirror publishes its XCD, then
    reads all of them) sits before a head's step-0 coarse gates, which wait
    for the mirrors' first words, and before a mirror publishes those: no
    interleaving deadlocks.  With the heads' check after their step-0 gates,
    every interleaving deadlocks (the mirrors wait for the heads' XCD words,
    the heads for the mirrors' words)."""
    assert not [sd for sd in range(40) if run(seed=sd, T=4)]
    assert all((run(seed=sd, T=4, heads_check_first=False) or "").startswith("deadlock") for sd in range(10))
