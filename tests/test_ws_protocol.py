"""Host model of the split kernels' workspace protocol (draw slots with generations, records of
two tagged 64-bit words), checked on the CPU against the property the look-back relies on:
when a call reads the record words it publishes, no word left there by an earlier call carries
the tag the reader expects for that word. A reader loads the two words of a record separately,
so a stale word with a current tag could pair with a current word of the other kind (this is
how per-slot generations once mixed a stale map into a carry after calls of another shape).

The model follows the kernels: a row call over N rows of P tiles draws from slots 0..N-1 and
writes records p*N + row; a column call over J columns in 64-column blocks draws from slots
0..ceil(J/64)-1 and writes records t*J + j; tags are (2*gen + 1, tag0 + N*M) for rows and
(2*gen + 2, tag0 + (4*J + kind)*M) for columns, M = 0x9e3779b1, all mod 2^32."""
import itertools
import random

import pytest

M = 0x9E3779B1
SLOTS = 1024
MASK32 = (1 << 32) - 1


class Workspace:
    def __init__(self, shared_generation: bool):
        self.gen = [0] * SLOTS
        self.words = {}  # (record index, word 0/1) -> tag
        self.shared = shared_generation

    def call(self, kind: str, n: int, P: int, backward: bool = False):
        """One split call: returns the (index, word, expected tag) reads that would accept a
        stale word. Every tile but the one at the row's (column's) output-side edge publishes
        its map: tiles 1..P-1 of a backward scan, 0..P-2 of a forward one."""
        used = n if kind == "row" else (n + 63) // 64
        slot_of = (lambda i: i) if kind == "row" else (lambda j: j // 64)
        parity = 1 if kind == "row" else 2
        tag_n = n if kind == "row" else 4 * n
        writes = []
        for i in range(n):
            g = self.gen[slot_of(i)]
            t0 = (2 * g + parity) & MASK32
            t1 = (t0 + tag_n * M) & MASK32
            for p in (range(1, P) if backward else range(P - 1)):
                idx = p * n + i
                writes.append((idx, t0, t1))
        bad = [(idx, w, t) for idx, t0, t1 in writes for w, t in ((0, t0), (1, t1))
               if self.words.get((idx, w)) == t]
        for idx, t0, t1 in writes:
            self.words[(idx, 0)] = t0
            self.words[(idx, 1)] = t1
        for s in range(used):
            self.gen[s] += 1
        if self.shared:
            g = self.gen[0] - 1
            for s in range(used, SLOTS):
                self.gen[s] = g + 1
        return bad


SEQUENCES = [
    # the sequence of the row-major reuse test: GAE (backward) then eligibility traces (forward)
    # on 64x8192, 3x5000, 64x8192 (1024-step tiles)
    [("row", 64, 8, True), ("row", 64, 8), ("row", 3, 5, True), ("row", 3, 5),
     ("row", 64, 8, True), ("row", 64, 8)],
    # GAE rows, time-major V-Trace columns, F-vector trace columns, forward rows, twice
    [("row", 64, 8, True), ("col", 200, 16, True), ("col", 640, 5), ("row", 3, 5)] * 2,
]


@pytest.mark.parametrize("seq", range(len(SEQUENCES)))
def test_per_slot_generations_let_stale_words_match(seq):
    """The protocol with a generation per slot: these call sequences leave a stale word with a
    current tag (the failure the shared generation removes)."""
    ws = Workspace(shared_generation=False)
    assert any(ws.call(*c) for c in SEQUENCES[seq])


@pytest.mark.parametrize("seq", range(len(SEQUENCES)))
def test_shared_generation_never_matches_a_stale_word(seq):
    ws = Workspace(shared_generation=True)
    for c in SEQUENCES[seq]:
        assert ws.call(*c) == []


def test_shared_generation_random_sequences():
    """Random mixes of row and column calls of many shapes on one workspace."""
    rng = random.Random(7)
    for _ in range(40):
        ws = Workspace(shared_generation=True)
        for _ in range(30):
            kind = "row" if rng.random() < 0.5 else "col"
            c = (kind, rng.randint(1, 80 if kind == "row" else 900), rng.randint(2, 12),
                 rng.random() < 0.5)
            assert ws.call(*c) == []
        # every slot stands at the same generation, the number of calls made
        assert len(set(ws.gen)) == 1 and ws.gen[0] == 30
