"""GPU parity of drafter play and regret bookkeeping against the oracle: choices bit-exact
(both sides take the sampling decision on left-to-right fp64 prefix sums) and the bookkeeping
sums bit-exact (fp64, the same order); an end-to-end stream of rounds across a regime switch."""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_20064_amd as hs
import synth

pytestmark = pytest.mark.gpu


def note(msg):
    print("\n[case] " + msg, flush=True)


@pytest.mark.parametrize("N", [1, 7, 64])
def test_play_matches_oracle(N):
    rng = np.random.default_rng(71 + N)
    B = 300
    w = rng.random((B, N))
    w[::7] = np.round(w[::7] * 3) / 3          # ties
    w[3] = 0.0                                  # no positive weight
    w[5] = 0.0
    w[5, N - 1] = 2.0                           # a point mass on the last drafter
    w[9] = w[9] / w[9].sum()                    # normalised
    u = rng.random(B)
    u[:4] = [0.0, 0.5, 1.0 - 2 ** -52, 0.25]
    note("play N=%d" % N)
    wd, ud = torch.from_numpy(w).cuda(), torch.from_numpy(u).cuda()
    for how in (hs.PLAY_ARGMAX, hs.PLAY_SAMPLE):
        got = hs.play(wd, how, ud).cpu().numpy()
        assert np.array_equal(got, oracle.play(w, how, u)), how


def test_regret_bookkeeping_matches_oracle():
    rng = np.random.default_rng(72)
    B, N = 9, 13
    st = hs.RegretState(B, N, "cuda")
    ref = oracle.Regret(B, N)
    note("regret bookkeeping, 20 updates")
    for r in range(20):
        L = int(rng.integers(1, 5))
        f = rng.random((L, B, N))
        pl = rng.integers(0, N, (L, B)).astype(np.int32)
        if r == 13:
            pl[0, 4] = N  # an invalid play: that query's sums become NaN
        eal = rng.random((B, N)) * 9
        st.update(torch.from_numpy(f).cuda(), torch.from_numpy(pl).cuda(), torch.from_numpy(eal).cuda())
        ref.update(f, pl, eal)
        torch.cuda.synchronize()
        assert np.array_equal(st.cum.cpu().numpy(), ref.cum, equal_nan=True)
        assert np.array_equal(st.played.cpu().numpy(), ref.played, equal_nan=True)
        assert np.array_equal(st.regret.cpu().numpy(), ref.regret, equal_nan=True)
        assert np.array_equal(st.eal_sum.cpu().numpy(), ref.eal_sum, equal_nan=True)


def test_play_and_regret_across_a_regime_switch():
    # the large-pool stream's regime switch (drafter quality order reverses), reduced to a
    # 4 x 16 x 8 round at V = 4096: play NormalHedge's argmax, then learn from the round
    w = synth.variant(synth.workloads()["large_pool_stream"], B=4, N=16, V=4096,
                      scales=synth.workloads()["large_pool_stream"].scales[:16], regime_switch=30)
    rounds = 60
    note("regime switch stream, %d rounds" % rounds)
    x0 = synth.generate(w, round=0)
    xd = torch.from_numpy(x0).view(torch.bfloat16).cuda()
    rnd = hs.Round(xd, V=w.V, temperature=w.temperature, mode=hs.SAMPLE, loss_kind=w.loss, eta=w.eta)
    reg = hs.RegretState(w.B, w.N, "cuda")
    ref = oracle.Regret(w.B, w.N)
    for r in range(rounds):
        if r:
            rnd.set_logits(torch.from_numpy(synth.generate(w, round=r)).view(torch.bfloat16).cuda())
        choice = hs.play(rnd.state.p, hs.PLAY_ARGMAX)  # before this round's update
        # the choice equals the oracle's on the same weights, bit for bit
        torch.cuda.synchronize()
        assert np.array_equal(choice.cpu().numpy(),
                              oracle.play(rnd.state.p.cpu().numpy(), 0).astype(np.int32)), r
        rnd.run()
        reg.update(rnd.loss, choice.view(1, -1), rnd.eal)
        torch.cuda.synchronize()
        ref.update(rnd.loss.cpu().numpy(), choice.cpu().numpy().reshape(1, -1), rnd.eal.cpu().numpy())
        assert np.array_equal(reg.regret.cpu().numpy(), ref.regret)
    assert np.array_equal(reg.eal_sum.cpu().numpy(), ref.eal_sum)
    # the learner recovers from the switch: per-round regret over the stream stays below the
    # loss gap between the best and worst drafters
    gap = (ref.cum.max(1) - ref.cum.min(1)) / rounds
    assert np.all(ref.regret / rounds < gap)
