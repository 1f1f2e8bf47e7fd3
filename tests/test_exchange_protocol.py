"""A CPU model of the batched kernel's exchange protocol (CPU only).

Heads and units of every group run the kernel's order of publishes and waits,
one read of one word per scheduling step, under random interleavings with
strongly skewed speeds.  The words carry the kernel's tags:

* y slices, partial logits, gate words (with the e gate's context term) and
  class words hold one parity bit of the step: a reader accepts a word whose
  bit matches and the model then checks that the word's full step is the one
  awaited (a parity match on another step is a misread);
* drawn samples sit in SS slots chosen by the step's tag modulo SS and carry
  16 bits of the tag: a reader whose slot already holds a later tag waits
  forever (a lost word, seen as a deadlock).

Both group modes are modelled: ALL (2 or 4 vectors per group: every head
reads every gate word of both halves in one poll at the start of the step and
draws every vector; one writer head per vector's sample word) and SLICE (8 vectors: head j evaluates its own slice of units and
the heads exchange y slices, vector v is owned by head v mod NH, which alone
gathers its partials, draws it and publishes its class words; the coarse gate
poll also waits for the first word of every unit and for the owners' classes
of the previous step, the fine poll for the classes of this step).  The units
wait for the drawn samples of step t - A of every lane of their utterance: at
the start of the step with a context lead A > 0 (before the halves of h), after
both halves with A = 0.  Sample words are published by idle lanes too.

What the model leaves out: values, the heads' LDS staging and barriers inside
a workgroup (a workgroup is one agent), the per-thread split of a poll (a
round's words are read one at a time, in order), memory-ordering effects of
the hardware (every write is visible to the next read), and the bounded waits'
clock.
"""
import random

import pytest


def run(mode="ALL", G=8, NH=3, NU=3, L=2, B=16, F=4, A=1, rows=12, SS=None, seed=0, idle_publish=True,
        max_ticks=4_000_000):
    rng = random.Random(seed)
    if SS is None:
        SS = 2
        while SS < 2 * A + 2:
            SS *= 2
    V = G * L
    T = rows + (B - 1) * (F + 1 + A)
    mem = {}
    pos = lambda v, t: t - (v % B) * (F + 1 + A)
    act = lambda v, t: 0 <= pos(v, t) < rows
    owner = (lambda v: (v % L) % NH) if mode == "SLICE" else (lambda v: (v % L) % NH)

    def pub(key, tag):
        return ("w", key, tag)

    def wait1(key, tag):   # one parity-tagged word
        return ("r1", key, tag)

    def wait16(key, tag):  # a sample word: 16 bits of tag in its slot
        return ("r16", key, tag)

    def samples(g, td):
        """The unit waits for the samples of step td of every lane of its utterance(s)."""
        if td < 0:
            return
        u0 = (g * L) // B
        nut = 1 if B >= L else L // B
        for vv in range(u0 * B, u0 * B + nut * B):
            if vv < V and (idle_publish or act(vv, td)):
                yield wait16(("S", vv // L, vv % L, (td + 1) % SS), td + 1)

    def head(g, j):
        for s in range(T):
            tag = s + 1
            own = [v for v in range(L) if owner(g * L + v) == j]
            # coarse gate words of every unit of the group (and, SLICE, every unit's first word
            # and the owners' classes of the previous step)
            for k in range(NU):
                yield wait1(("GATE", g, k), tag)
            if mode == "SLICE" and s > 0:
                for v in range(L):
                    yield wait1(("CC", g, v), tag - 1)
                    yield wait1(("CF", g, v), tag - 1)
            yield pub(("YC", g, j), tag)
            if mode == "SLICE":
                for jj in range(NH):
                    if jj != j:
                        yield wait1(("YC", g, jj), tag)
            yield pub(("PC", g, j), tag)
            for jj in range(NH):                     # (ALL: every vector; SLICE: the owned ones)
                if mode == "ALL" or own:
                    yield wait1(("PC", g, jj), tag)
            if mode == "SLICE":
                for v in own:
                    yield pub(("CC", g, v), tag)
            # fine: SLICE polls its gate words (published with the coarse ones) with this
            # step's classes; ALL read them with the coarse words above
            if mode == "SLICE":
                for k in range(NU):
                    yield wait1(("GATE", g, k), tag)
                for v in range(L):
                    yield wait1(("CC", g, v), tag)
            yield pub(("YF", g, j), tag)
            if mode == "SLICE":
                for jj in range(NH):
                    if jj != j:
                        yield wait1(("YF", g, jj), tag)
            yield pub(("PF", g, j), tag)
            for jj in range(NH):
                if mode == "ALL" or own:
                    yield wait1(("PF", g, jj), tag)
            for v in range(L):
                if owner(g * L + v) == j:
                    if mode == "SLICE":
                        yield pub(("CF", g, v), tag)
                    if idle_publish or act(g * L + v, s):
                        yield pub(("S", g, v, tag % SS), tag)

    def unit(g, k):
        yield pub(("GATE", g, k), 1)
        for t in range(T - 1):
            tag = t + 1
            if A > 0:
                yield from samples(g, t - A)
            for j in range(NH):
                yield wait1(("YC", g, j), tag)
            for j in range(NH):
                yield wait1(("YF", g, j), tag)
            if A == 0:
                yield from samples(g, t)
            yield pub(("GATE", g, k), tag + 1)

    agents = [head(g, j) for g in range(G) for j in range(NH)] + [unit(g, k) for g in range(G) for k in range(NU)]
    speed = [rng.random() ** 4 + 0.002 for _ in agents]     # some agents hundreds of times slower
    cur = [next(a) for a in agents]
    live = set(range(len(agents)))

    def ready(i):
        kind, key, tag = cur[i]
        if kind == "w":
            return True
        x = mem.get(key, 0)
        return (x & 1) == (tag & 1) if kind == "r1" else (x & 0xFFFF) == (tag & 0xFFFF)

    for _ in range(max_ticks):
        if not live:
            return None
        rd = [i for i in live if ready(i)]
        if not rd:
            stuck = [(cur[i], mem.get(cur[i][1], 0)) for i in sorted(live)][:4]
            return f"deadlock (a word lost or never written): {stuck}"
        i = rng.choices(rd, weights=[speed[x] for x in rd])[0]
        kind, key, tag = cur[i]
        if kind == "w":
            mem[key] = tag
        elif mem.get(key, 0) != tag:
            return f"misread: {key} awaited at step tag {tag}, holds {mem.get(key, 0)}"
        try:
            cur[i] = next(agents[i])
        except StopIteration:
            live.discard(i)
    return "ran out of ticks"


@pytest.mark.parametrize("mode,G,L", [("ALL", 8, 2), ("ALL", 4, 4), ("SLICE", 2, 8)])
@pytest.mark.parametrize("A", [0, 1, 2])
def test_exchange_protocol_has_no_lost_or_misread_word(mode, G, L, A):
    """Random interleavings, skewed speeds: every awaited word is read with
    the step it was awaited for, and nothing waits forever (B = 16 lanes of
    one utterance over the groups, horizon 4, the kernel's slot count)."""
    fails = [(sd, e) for sd in range(6) for e in [run(mode, G=G, L=L, A=A, seed=sd)] if e]
    assert not fails, fails[:2]


def test_the_model_catches_a_reused_sample_slot():
    """The model is not blind: with too few sample slots (SS = 2 at A = 1) or
    without idle lanes publishing, some interleaving loses a sample word."""
    assert any(run("ALL", A=1, SS=2, seed=sd) for sd in range(40))
    assert any(run("ALL", A=1, idle_publish=False, seed=sd) for sd in range(40))
