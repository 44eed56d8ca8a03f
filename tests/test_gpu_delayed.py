"""GPU parity of hs_delayed_update (token-level length loss with delayed feedback, QFI-D with
Hedge and NormalHedge) against the float64 oracle, through the C ABI.

Tolerances: window losses within 1e-12 absolute (fp64 on both sides, from the same fp32
feedback); Hedge and NormalHedge weights within 1e-5 absolute, as for the round's learners."""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_20064_amd as hs

pytestmark = pytest.mark.gpu

LOSS_TOL = 1e-12
W_TOL = 1e-5


def note(msg):
    print("\n[case] " + msg, flush=True)


def _run(B, N, K, rounds, eta, mode, seed, max_count=None, hybrid=0):
    rng = np.random.default_rng(seed)
    st = hs.DelayedState(B, N, K, "cuda")
    q = oracle.QfiD(B, N, K, eta, hybrid=hybrid)
    mc = K if max_count is None else max_count
    for r in range(rounds):
        if mode == hs.SAMPLE:
            g32 = rng.random((B, N, K)).astype(np.float32)
            gd = torch.from_numpy(g32).cuda()
        else:
            g32 = (rng.random((B, N, K)) < 0.7).astype(np.uint8)
            gd = torch.from_numpy(g32).cuda()
        cnt = rng.integers(0, mc + 1, B).astype(np.int32)
        hs.delayed_update(st, gd, torch.from_numpy(cnt).cuda(), eta, mode=mode,
                          hybrid_tokens=hybrid)
        used = q.push(g32.astype(np.float64), cnt)
        torch.cuda.synchronize()
        nl = st.nloss.cpu().numpy()
        ls = st.loss.cpu().numpy()
        for b in range(B):
            assert nl[b] == used[b].shape[0], (r, b)
            if nl[b]:
                assert np.abs(ls[:nl[b], b, :] - used[b]).max() <= LOSS_TOL, (r, b)
        assert np.abs(st.learners.w.cpu().numpy() - q.w).max() <= W_TOL, r
        assert np.abs(st.learners.p.cpu().numpy() - q.p).max() <= W_TOL, r
        assert np.allclose(st.learners.c.cpu().numpy(), q.c, rtol=1e-9, atol=0), r
        clock = st.clock.cpu().numpy()
        assert np.array_equal(clock[:, 1], np.array(q.done)), r
    return st


@pytest.mark.parametrize("mode", [hs.SAMPLE, hs.GREEDY])
def test_delayed_small_ragged_counts(mode):
    note("B=3 N=5 K=4, 40 rounds of ragged counts, mode %d" % mode)
    _run(3, 5, 4, 40, 0.4, mode, seed=1)


def test_delayed_window_one_and_full_pool():
    note("K=1 (no delay beyond the token) and N=64, K=8, B=32, 12 rounds")
    _run(2, 7, 1, 20, 0.3, hs.SAMPLE, seed=2)
    _run(32, 64, 8, 12, 0.182404, hs.SAMPLE, seed=3)


def test_delayed_no_window_leaves_state_and_counts_clamp():
    note("calls that complete no window leave the learners as they are; counts clamp to [0, K]")
    B, N, K = 2, 4, 6
    st = hs.DelayedState(B, N, K, "cuda")
    g = torch.rand((B, N, K), device="cuda")
    for cnt in ([2, 0], [3, 5]):  # 5 and 5 tokens: no window of 6 yet
        hs.delayed_update(st, g, torch.tensor(cnt, dtype=torch.int32, device="cuda"), 0.5)
    torch.cuda.synchronize()
    assert st.nloss.cpu().tolist() == [0, 0]
    assert torch.all(st.learners.w == 1.0 / N) and torch.all(st.learners.R == 0)
    assert st.clock.cpu().tolist() == [[5, 0], [5, 0]]
    hs.delayed_update(st, g, torch.tensor([-3, 99], dtype=torch.int32, device="cuda"), 0.5)
    torch.cuda.synchronize()
    assert st.clock.cpu().tolist() == [[5, 0], [11, 6]]  # clamped to 0 and K
    assert st.nloss.cpu().tolist() == [0, 6]


def test_delayed_chunking_invariance():
    note("the same token stream in two chunkings: same window losses and NormalHedge state")
    B, N, K, T = 2, 6, 5, 37
    rng = np.random.default_rng(4)
    stream = rng.random((B, T, N)).astype(np.float32)
    outs = []
    for split_seed in (5, 6):
        srng = np.random.default_rng(split_seed)
        st = hs.DelayedState(B, N, K, "cuda")
        pos = [0, 0]
        all_losses = [[], []]
        while min(pos) < T:
            cnt = [min(int(srng.integers(0, K + 1)), T - pos[b]) for b in range(B)]
            g = np.zeros((B, N, K), np.float32)
            for b in range(B):
                g[b, :, :cnt[b]] = stream[b, pos[b]:pos[b] + cnt[b]].T
            hs.delayed_update(st, torch.from_numpy(g).cuda(),
                              torch.tensor(cnt, dtype=torch.int32, device="cuda"), 0.7)
            torch.cuda.synchronize()
            nl = st.nloss.cpu().numpy()
            ls = st.loss.cpu().numpy()
            for b in range(B):
                all_losses[b].append(ls[:nl[b], b].copy())
                pos[b] += cnt[b]
        outs.append((st, [np.concatenate(x) for x in all_losses]))
    (s1, l1), (s2, l2) = outs
    for b in range(B):
        assert l1[b].shape == (T - K + 1, N) and np.array_equal(l1[b], l2[b])
    assert torch.equal(s1.learners.R, s2.learners.R) and torch.equal(s1.learners.p, s2.learners.p)
    assert torch.equal(s1.learners.c, s2.learners.c)
    assert torch.allclose(s1.learners.w, s2.learners.w, rtol=0, atol=1e-12)


@pytest.mark.parametrize("hybrid", [3, 7, 1000])
def test_delayed_hybrid_losses(hybrid):
    # acceptance losses for the first H tokens of each stream, then window length losses
    note("hybrid H=%d, B=4 N=6 K=5, 30 rounds" % hybrid)
    _run(4, 6, 5, 30, 0.5, hs.SAMPLE, seed=11, hybrid=hybrid)


def test_update_cadence_matches_per_round_updates_at_every_update():
    rng = np.random.default_rng(12)
    B, N, K, rounds = 3, 7, 4, 40
    gam = [torch.from_numpy(rng.random((B, N, K)).astype(np.float32)).cuda() for _ in range(rounds)]
    cnt = [torch.from_numpy(rng.integers(0, K + 1, B).astype(np.int32)).cuda() for _ in range(rounds)]
    note("update cadence: warm-up 6, batches of 12, hybrid 5")
    every = hs.DelayedState(B, N, K, "cuda")
    batched = hs.DelayedState(B, N, K, "cuda")
    cad = hs.UpdateCadence(batched, 0.5, warmup=6, batch=12, hybrid_tokens=5)
    prev_w = batched.learners.w.clone()
    for r in range(rounds):
        hs.delayed_update(every, gam[r], cnt[r], 0.5, hybrid_tokens=5)
        updated = cad.push(gam[r], cnt[r])
        torch.cuda.synchronize()
        assert updated == cad.due(r)
        if updated:  # the same kernel calls in the same order: the same bits
            for f in ("logw", "w", "R", "p", "c"):
                assert torch.equal(getattr(batched.learners, f), getattr(every.learners, f)), (r, f)
            prev_w = batched.learners.w.clone()
        else:
            assert torch.equal(batched.learners.w, prev_w), r
    assert [r for r in range(rounds) if cad.due(r)] == [0, 1, 2, 3, 4, 5, 17, 29]
