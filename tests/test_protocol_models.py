"""CPU models of the two cross-workgroup protocols of the epoch kernels, run under random
interleavings of their waves (host only; no GPU).

* The staged hot-set epoch: stager waves (other CUs) stage batches into a ring of R records and
  write each batch's results out; loader waves of the hot workgroup publish results, take records
  (read ahead when the tag was already seen) and hand buffers to the consumer waves.  The model
  follows the kernel's order of waits and flag writes and reads flag words ahead the way the loader
  does.  Checked: no interleaving deadlocks (for 1 to 192 stager waves, one to four consumers, rings
  of 2 to 64 records), every record a loader takes is its batch's, every result a stager reads is its
  batch's, and every batch is written out exactly once.
* The split epoch: workgroups claim chunks of units in order and process them in order; a SCATTER
  unit waits for the GATHER slots of its coordinate.  Checked: no deadlock for any number of
  workgroups and chunk sizes, and every part of a coordinate takes the same step (the sum of all its
  GATHER partials).
"""
import random

import pytest


# ------------------------------------------------------------------------------------------ staged

class Staged:
    """One epoch of nb batches: G stager waves, NP loaders (buffer q takes batches q, q + NP, ...),
    NC consumers (batch b goes to consumer b mod NC), a ring of R records and R result slots."""

    def __init__(self, nb, R, G, NC, seed):
        self.rng = random.Random(seed)
        self.nb, self.R, self.NC = nb, R, NC
        self.NP = 12 - NC
        self.tag = [0] * R        # record slot s: last batch published there, + 1
        self.loaded = [0] * R     # record slot s: last batch a loader took from it, + 1
        self.rec = [None] * R     # the batch whose record is in slot s
        self.res = [0] * R        # result slot s: last batch whose results were published, + 1
        self.res_read = [0] * R   # result slot s: last batch whose stager read its results, + 1
        self.ready = [0] * self.NP
        self.freed = [0] * self.NP
        self.claim = 0
        self.written = []
        self.stagers = [dict(b=None, ph=0) for _ in range(G)]
        self.loaders = [dict(b=q, ph=0, pre=False, tag_seen=0, tag_ahead=0, res_seen=0, held=None, published=True)
                        for q in range(self.NP)]
        for q, L in enumerate(self.loaders):
            if q + self.NP < nb:
                L["tag_ahead"] = self.tag[(q + self.NP) % R]
        self.consumers = [c for c in range(NC)]

    # Each step function returns True if the actor made progress.
    def stager(self, S):
        R = self.R
        if S["b"] is None:
            if self.claim >= self.nb:
                return False
            S["b"], S["ph"] = self.claim, 0
            self.claim += 1
            return True
        b = S["b"]
        s = b % R
        if S["ph"] == 0:  # wait until the slot's previous batch has been taken, then stage and publish
            if b >= R and self.loaded[s] != b - R + 1:
                return False
            self.rec[s] = b
            self.tag[s] = b + 1
            S["ph"] = 1
            return True
        # wait for this batch's results, mark them read, write the batch out
        if self.res[s] != b + 1:
            return False
        self.res_read[s] = b + 1
        self.written.append(b)
        S["b"] = None
        return True

    def take_record(self, L, b):
        s = b % self.R
        assert self.tag[s] == b + 1 and self.rec[s] == b, "a loader took a record that is not its batch's"
        L["held"] = b

    def loader(self, q):
        L = self.loaders[q]
        R, NP, nb = self.R, self.NP, self.nb
        b = L["b"]
        if b >= nb + NP:
            return False
        n = b // NP
        c = b - NP
        if L["ph"] == 0:  # the consumer has finished the buffer's previous batch
            if (n > 0 or b < nb) and self.freed[q] != n:
                return False
            L["ph"], L["published"] = 1, n == 0
            return True
        if L["ph"] == 1:  # the previous batch's result slot must be free before its results are published
            if n > 0 and c >= R:
                s = c % R
                if L["res_seen"] != c - R + 1 and self.res_read[s] != c - R + 1:
                    return False
            L["ph"] = 2
            return True
        if L["ph"] == 2:  # the record: read ahead, or wait for its tag now (results published first)
            if b < nb and not L["pre"]:
                s = b % R
                if L["tag_seen"] != b + 1:
                    if not L["published"]:
                        self.publish(L, c)
                        return True
                    if self.tag[s] != b + 1:
                        return False
                self.take_record(L, b)
            if b < nb:
                assert L["held"] == b
                self.ready[q] = n + 1  # image written, buffer handed over
                b2 = b + NP
                L["pre"] = b2 < nb and L["tag_ahead"] == b2 + 1
                if L["pre"]:
                    self.take_record(L, b2)
            L["ph"] = 3
            return True
        # ph 3: publish the results if not done yet; free this record's slot; read the flag words ahead.
        if not L["published"]:
            self.publish(L, c)
        if b >= nb:
            L["b"] = nb + NP  # done
            return True
        b2, b3 = b + NP, b + 2 * NP
        self.loaded[b % R] = b + 1
        L["tag_seen"] = self.tag[b2 % R] if (b2 < nb and not L["pre"]) else 0
        L["tag_ahead"] = self.tag[b3 % R] if b3 < nb else 0
        L["res_seen"] = self.res_read[b % R] if b >= R else 0
        L["b"], L["ph"] = b2, 0
        return True

    def publish(self, L, c):
        s = c % self.R
        assert c < self.R or self.res_read[s] == c - self.R + 1, "results overwritten before they were read"
        self.res[s] = c + 1
        L["published"] = True

    def consumer(self, i):
        b = self.consumers[i]
        if b >= self.nb:
            return False
        p, n = b % self.NP, b // self.NP
        if self.ready[p] != n + 1:
            return False
        self.freed[p] = n + 1
        self.consumers[i] = b + self.NC
        return True

    def run(self):
        actors = ([lambda S=S: self.stager(S) for S in self.stagers] +
                  [lambda q=q: self.loader(q) for q in range(self.NP)] +
                  [lambda i=i: self.consumer(i) for i in range(self.NC)])
        while True:
            order = list(range(len(actors)))
            self.rng.shuffle(order)
            progressed = False
            for k in order:
                # take a random number of steps of this actor (models uneven wave speeds)
                for _ in range(self.rng.randint(1, 3)):
                    if actors[k]():
                        progressed = True
                    else:
                        break
            if not progressed:
                break
        return sorted(self.written)


@pytest.mark.parametrize("NC", [1, 2, 3, 4])
@pytest.mark.parametrize("R", [2, 5, 10, 64])
@pytest.mark.parametrize("G", [1, 3, 192])
def test_staged_protocol_completes_without_stale_records(NC, R, G):
    for nb in (1, 11, 64, 65, 300):
        for seed in range(3):
            m = Staged(nb, R, G, NC, seed)
            written = m.run()
            assert written == list(range(nb)), (nb, R, G, NC, seed, len(written))
            assert all(L["b"] >= nb for L in m.loaders)
            assert all(b >= nb for b in m.consumers)


def test_staged_model_detects_a_missing_wait():
    # The same model with the loader's result-slot wait removed must fail, so the checks above can
    # see a protocol mistake.
    class NoResWait(Staged):
        def loader(self, q):
            L = self.loaders[q]
            if L["ph"] == 1:
                L["ph"] = 2
                return True
            return super().loader(q)

        def publish(self, L, c):
            self.res[c % self.R] = c + 1  # no check that the slot's previous results were read
            L["published"] = True

    failed = False
    for seed in range(20):
        m = NoResWait(200, 2, 192, 2, seed)
        if m.run() != list(range(200)):
            failed = True
            break
    assert failed


def test_staged_model_detects_waiting_for_a_tag_while_holding_results():
    # Waiting for the next record's tag before publishing the results it holds deadlocks when the
    # stager waves are few: the order the kernel follows matters.
    class TagFirst(Staged):
        def loader(self, q):
            L = self.loaders[q]
            b = L["b"]
            if L["ph"] == 2 and b < self.nb and not L["pre"] and L["tag_seen"] != b + 1 and not L["published"]:
                if self.tag[b % self.R] != b + 1:
                    return False  # waits for the tag first
            return super().loader(q)

    assert any(TagFirst(200, 64, 1, 2, seed).run() != list(range(200)) for seed in range(5))


# ------------------------------------------------------------------------------------------- split

def split_units(lens, part):
    """Units in permutation order: (kind, coordinate, part index, parts, first GATHER unit index)."""
    units = []
    for c, ln in enumerate(lens):
        if ln <= part:
            units.append(("FULL", c, 0, 1, None))
        else:
            k = -(-ln // part)
            g0 = len(units)
            units += [("GATHER", c, i, k, g0) for i in range(k)]
            units += [("SCATTER", c, i, k, g0) for i in range(k)]
    return units


def run_split(lens, part, n_wg, chunk, seed, in_order=True):
    rng = random.Random(seed)
    units = split_units(lens, part)
    partial = [None] * len(units)   # GATHER slots
    steps = {}                      # coordinate -> steps taken by its SCATTER parts
    done = [False] * len(units)
    queue = [0]
    wgs = [[] for _ in range(n_wg)]  # each workgroup's claimed, unfinished units, in order

    def step(w):
        if not wgs[w]:
            if queue[0] >= len(units):
                return False
            u0 = queue[0]
            queue[0] = min(len(units), u0 + chunk)
            wgs[w] = list(range(u0, queue[0]))
            return True
        u = wgs[w][0] if in_order else wgs[w][-1]
        kind, c, i, k, g0 = units[u]
        if kind == "GATHER":
            partial[u] = (c, i, rng.random())  # this part's contribution to the inner product
        elif kind == "SCATTER":
            slots = partial[g0:g0 + k]
            if any(p is None for p in slots):
                return False
            assert [p[:2] for p in slots] == [(c, j) for j in range(k)]
            steps.setdefault(c, []).append(sum(p[2] for p in slots))  # fixed order: the same in every part
        done[u] = True
        wgs[w].remove(u)
        return True

    while True:
        order = list(range(n_wg))
        rng.shuffle(order)
        if not any([step(w) for w in order]):
            break
    if not all(done):
        return False  # deadlock: some unit never finished
    parts = {u[1]: u[3] for u in units if u[0] == "SCATTER"}
    assert sorted(steps) == sorted(parts)
    for c, s in steps.items():
        assert len(s) == parts[c]
        assert len(set(s)) == 1, "the parts of one coordinate took different steps"
    return True


@pytest.mark.parametrize("n_wg", [1, 2, 7, 64])
@pytest.mark.parametrize("chunk", [1, 3, 16])
def test_split_protocol_progress_and_identical_steps(n_wg, chunk):
    rng = random.Random(n_wg * 100 + chunk)
    for seed in range(4):
        lens = [rng.choice([1, 5, 64, 65, 300, 1000]) for _ in range(40)]
        assert run_split(lens, 64, n_wg, chunk, seed), "deadlock"


def test_split_model_detects_out_of_order_units():
    # A workgroup that took its claimed units out of order could wait on a GATHER unit it holds
    # itself: the model must report that deadlock.
    lens = [300] * 8
    assert not run_split(lens, 64, 1, 16, 0, in_order=False)
