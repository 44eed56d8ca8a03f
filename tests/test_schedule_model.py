"""The team kernel's row-set schedule, modelled on the host (CPU only).

A team of the pipelined kernel runs its items three deep: item j's min-sum, item j + 1's
statistics, item j + 2's loads. Its units are blocks: a (query, position) group's nsub row sets
when the groups outnumber the teams four times over, single row sets otherwise. Its first kB
blocks are fixed (blocks T, T + teams, ...; at least three items), and an item that starts a
later block is claimed three items ahead from a device-wide counter whose values start past
every team's fixed blocks. This model follows the kernel's successor rule step by step, with
the teams' iterations interleaved at random, and checks that every row set is taken exactly
once and that no item of the first three needs a claim.
"""
import random

import pytest


def schedule(nsets, nsub, teams, seed):
    rnd = random.Random(seed)
    blocked = nsub > 1 and nsets >= 4 * teams * nsub
    bsz = nsub if blocked else 1
    nblocks = nsets // nsub if blocked else nsets
    kB = -(-3 // bsz) if blocked else 3
    dyn = kB * teams < nblocks
    counter = 0
    taken = []
    claim = object()

    class Team:
        def __init__(self, T):
            self.T, self.nblk = T, 0

        def first(self, bl):
            return bl * bsz if bl < nblocks else nsets

        def successor(self, s):
            if s >= nsets:
                return nsets
            if blocked and (s + 1) % nsub != 0:
                return s + 1
            if self.nblk < kB:
                v = self.first(self.T + self.nblk * teams)
                self.nblk += 1
                return v
            return claim if dyn else nsets

    live = []
    for T in range(teams):
        tm = Team(T)
        tm.set = tm.first(T)
        tm.nblk = 1
        tm.set1 = tm.successor(tm.set)
        tm.set2 = tm.successor(tm.set1)
        assert tm.set1 is not claim and tm.set2 is not claim
        live.append(tm)
    while live:
        tm = rnd.choice(live)
        if tm.set >= nsets:
            live.remove(tm)
            continue
        s3 = tm.successor(tm.set2)
        if s3 is claim:
            s3 = tm.first(kB * teams + counter)
            counter += 1
        taken.append(tm.set)
        if tm.set1 >= nsets:
            live.remove(tm)
            continue
        tm.set, tm.set1, tm.set2 = tm.set1, tm.set2, s3
    return blocked, sorted(taken)


@pytest.mark.parametrize("nsub", [1, 2, 3, 8])
@pytest.mark.parametrize("groups", [1, 2, 3, 5, 8, 40, 100, 256, 1024])
def test_every_row_set_taken_once(groups, nsub):
    nsets = groups * nsub
    for teams in (1, 2, 3, 7, 10, 64):
        if teams > nsets:
            continue
        for seed in range(3):
            blocked, taken = schedule(nsets, nsub, teams, seed)
            assert taken == list(range(nsets)), (groups, nsub, teams, seed)
            assert blocked == (nsub > 1 and groups >= 4 * teams)


def test_the_large_pool_and_the_draft_tree_are_blocked():
    # 256 groups of 8 row sets and 1024 groups of 2 row sets, 10 teams of 75 workgroups
    assert schedule(256 * 8, 8, 10, 0)[0]
    assert schedule(1024 * 2, 2, 10, 0)[0]
