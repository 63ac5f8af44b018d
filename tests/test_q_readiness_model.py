"""Model check, on the CPU, of the readiness rule between the per-sample kernel's tile
workgroups and its sequential workgroup (the chunked regrouping of the per-sample SGD step,
eq. (2)-(13), section "Fundamentals").

Model: nrb tiles each publish Q_0 and Q_1 at step 0, then at step s >= 1 wait until the
errors of chunk s-1 exist and publish Q_{s+1}; every publish adds 1 to a counter.  The
sequential side takes the chunks in order: it accepts Q_c by the counter rule, then produces
chunk c's errors.  Random interleavings of single publishes and single counter reads check
that the rule in use (one counter per chunk parity, complete at nrb (c // 2 + 1)) never
accepts a Q_c that some tile has not published, and that the single counter with the
threshold nrb (c + 1) does accept one, so the check can tell the two apart.
"""
import random


def run(nrb, nchk, per_parity, rng):
    """One random interleaving; returns True if an incomplete Q_c was accepted."""
    pub = [0] * nrb          # Q's published per tile (tile i has Q_0 .. Q_{pub[i]-1})
    counters = [0, 0]        # per-parity counters (per_parity) or counters[0] alone
    dready = 0               # chunks whose errors exist
    c = 0                    # chunk the sequential side waits for
    while c < nchk:
        movable = [i for i in range(nrb) if pub[i] < nchk and (pub[i] < 2 or dready >= pub[i] - 1)]
        if movable and rng.random() < 0.7:
            i = rng.choice(movable)
            q = pub[i]
            pub[i] += 1
            counters[q & 1 if per_parity else 0] += 1
            continue
        if per_parity:
            ready = counters[c & 1] >= nrb * (c // 2 + 1)
        else:
            ready = counters[0] >= nrb * (c + 1)
        if ready:
            if any(p <= c for p in pub):
                return True
            dready = c + 1
            c += 1
        elif not movable:
            raise AssertionError("model deadlock")
    return False


def test_per_parity_rule_never_accepts_an_incomplete_q():
    rng = random.Random(20230419)
    for _ in range(4000):
        nrb, nchk = rng.randint(1, 6), rng.randint(1, 9)
        assert not run(nrb, nchk, True, rng)


def test_single_counter_rule_accepts_an_incomplete_q():
    rng = random.Random(7)
    bad = sum(run(rng.randint(2, 6), rng.randint(2, 9), False, rng) for _ in range(4000))
    assert bad > 0
