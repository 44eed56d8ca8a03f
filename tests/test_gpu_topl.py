"""GPU parity of hs_eval_topl (Theorem 2, EAGLE's top-L acceptance mass) against the oracle.

Tolerances: the children (Top_L in rank order) and the greedy hit are bit-exact, since both
sides rank the same stored logits by value and then by lower index; gamma, a sum of at most 32
fp32 softmax terms against fp32 slice normalisers, within 2e-5 absolute (the alpha tolerance).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_20064_amd as hs
import synth

pytestmark = pytest.mark.gpu

GAMMA_TOL = 2e-5
WL = synth.workloads()


def note(msg):
    print("\n[case] " + msg, flush=True)


def to_dev(x: np.ndarray) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x))
    if x.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.cuda()


def run_topl(x, L, V=None, T=1.0, mode=hs.SAMPLE, children=True):
    out = hs.eval_topl(to_dev(x), L=L, V=V, temperature=T, mode=mode,
                       want_gamma=(mode == hs.SAMPLE), want_hit=True, want_children=children)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def check(x, L, V=None, T=1.0, mode=hs.SAMPLE, groups=None):
    """GPU on the whole [R][B][K][ld] tensor; the oracle on `groups` ((b, k) list, None = all)."""
    got = run_topl(x, L, V=V, T=T, mode=mode)
    if groups is None:
        B, K = x.shape[1], x.shape[2]
        groups = [(b, k) for b in range(B) for k in range(K)]
        ref = oracle.topl(x, L, V=V, T=T, want_mass=(mode == hs.SAMPLE))
        ref = {key: v.reshape((B * K,) + v.shape[2:]) for key, v in ref.items()}
    else:
        sub = np.stack([x[:, b, k] for (b, k) in groups], axis=1)
        ref = oracle.topl(sub, L, V=V, T=T, want_mass=(mode == hs.SAMPLE))
    worst = 0.0
    for gi, (b, k) in enumerate(groups):
        assert np.array_equal(got["children"][b, :, k], ref["idx"][gi]), (b, k)
        assert np.array_equal(got["hit"][b, :, k], ref["hit"][gi]), (b, k)
        if mode == hs.SAMPLE:
            worst = max(worst, float(np.abs(got["gamma"][b, :, k] - ref["gamma"][gi]).max()))
    assert worst <= GAMMA_TOL, worst
    return got


@pytest.mark.parametrize("dtype", [synth.BF16, synth.F32, synth.F16])
@pytest.mark.parametrize("N", [1, 3, 8, 11])
@pytest.mark.parametrize("L", [1, 10, 32])
def test_topl_small_ragged(dtype, N, L):
    # several slices and a ragged tail (V not a multiple of the 16-byte vector either)
    w = synth.variant(WL["qwen3_8b_single"], B=2, K=3, N=N, V=5003, ld=5008, dtype=dtype,
                      scales=[0.3 + 0.2 * i for i in range(N)], permute=False)
    note("small ragged dtype=%d N=%d L=%d" % (dtype, N, L))
    check(synth.generate(w), L, V=w.V, T=0.7)


def test_topl_greedy_mode_hits_only():
    w = synth.variant(WL["qwen3_8b_single"], B=2, K=4, V=9000)
    x = synth.generate(w)
    x[3] = x[0]  # a drafter identical to the target: every hit is 1
    note("greedy hits")
    got = check(x, 10, mode=hs.GREEDY)
    assert np.all(got["hit"][:, 2, :] == 1)


def _bf16(a):
    u = np.asarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def test_topl_ties_signed_zeros_and_infinities():
    rng = np.random.default_rng(21)
    V = 6000
    R, B, K = 7, 1, 4
    z = rng.normal(0, 2, (R, B, K, V)).astype(np.float32)
    z[1] = np.round(z[1])                 # few levels: ties across slices
    z[2] = 0.0                            # one level: Top_L is the first L tokens
    z[2, :, :, ::3] = -0.0                # ... with signed zeros among them
    z[3] = -np.inf                        # fewer than L finite logits, all in the tail slice
    z[3, :, :, 5990:5995] = rng.normal(0, 1, 5).astype(np.float32)
    z[4, :, :, :] = -np.inf               # no finite logit at all
    z[0, :, 1, ::2] = -np.inf             # a target with masked tokens
    z[5] = z[0]                           # a copy of the target
    z[6] = -z[0]
    for x in (z, _bf16(z), z.astype(np.float16)):
        note("ties, zeros, infinities dtype=%s" % x.dtype)
        for L in (1, 7, 32):
            check(x, L, T=0.9)


def test_topl_full_size_single_query():
    w = WL["qwen3_8b_single"]
    note("qwen3_8b_single full, L=10")
    check(synth.generate(w), 10, T=w.temperature)


def test_topl_large_pool_every_group():
    # the large pool's full shape (B32 N64 K8 V151936 bf16), every (query, drafter, position)
    w = WL["large_pool_stream"]
    note("large_pool_stream full shape, every group, L=10")
    x = synth.generate(w)
    check(x, 10, T=w.temperature)


def test_topl_longest_rows_and_crowded_merge():
    # V at the limit (512 slices). The first token of every slice is the largest, so the merge
    # sees more than its LDS holds above the first threshold and searches the lists in place.
    V = 2048 * 512
    rng = np.random.default_rng(22)
    z = rng.normal(0, 1, (2, 1, 1, V)).astype(np.float32)
    z[1, 0, 0, ::2048] = 100.0
    x = _bf16(z)
    note("V=%d crowded merge" % V)
    got = check(x, 32, T=1.0)
    assert list(got["children"][0, 0, 0]) == [2048 * s for s in range(32)]


def test_topl_deterministic_and_workspace_reuse():
    w = synth.variant(WL["qwen3_8b_single"], V=40000)
    x = to_dev(synth.generate(w))
    note("determinism")
    a = hs.eval_topl(x, L=10, want_children=True)
    b = hs.eval_topl(x, L=10, want_children=True)
    torch.cuda.synchronize()
    assert torch.equal(a["gamma"], b["gamma"]) and torch.equal(a["children"], b["children"])


@pytest.mark.parametrize("L", [2, 3])
def test_topl_candidate_list_overflow(L):
    # In every slice the first lane pair holds the largest values and the second pair the next
    # ones, so more keys reach the pair threshold than the slice's candidate list holds (L * 32
    # for bf16, L * 16 for fp32) and the slice kernel searches its registers instead.
    rng = np.random.default_rng(23)
    V = 8192
    z = rng.normal(0, 1, (3, 1, 2, V)).astype(np.float32)
    for base in range(0, V, 2048):
        for q in range(4):  # bf16 layout: lane l holds tokens q*512 + 8l .. 8l+7
            z[1, :, :, base + q * 512: base + q * 512 + 16] = 100.0
            z[1, :, :, base + q * 512 + 16: base + q * 512 + 32] = 50.0
    for base in range(0, V, 1024):
        for q in range(4):  # fp32 layout: lane l holds tokens q*256 + 4l .. 4l+3
            z[2, :, :, base + q * 256: base + q * 256 + 8] = 100.0
            z[2, :, :, base + q * 256 + 8: base + q * 256 + 16] = 50.0
    for x in (_bf16(z), z):
        note("candidate overflow L=%d dtype=%s" % (L, x.dtype))
        got = check(x, L, T=1.0)
        assert list(got["children"][0, 0, 0]) == list(range(L))


def test_topl_merge_long_candidate_list():
    # every slice holds the same 32 large values, so about 31 of each slice's 32 listed keys
    # reach the merge's first threshold: some 500 candidates, searched bitwise in LDS
    rng = np.random.default_rng(24)
    V = 16 * 2048
    z = rng.normal(0, 1, (2, 1, 1, V)).astype(np.float32)
    for s in range(16):
        z[1, 0, 0, s * 2048 + 64 * np.arange(32)] = 100.0 + np.arange(32)
    x = _bf16(z)
    note("merge long candidate list")
    got = check(x, 32, T=1.0)
    want = [s * 2048 + 64 * 31 for s in range(16)] + [s * 2048 + 64 * 30 for s in range(16)]
    assert list(got["children"][0, 0, 0]) == want


def test_topl_fp32_full_vocabulary():
    w = synth.variant(WL["qwen3_8b_single"], K=2, N=3, dtype=synth.F32,
                      scales=[0.4, 0.8, 1.6], permute=False)
    note("fp32 V=151936, N=3, K=2, L=10 and 32")
    x = synth.generate(w)
    for L in (10, 32):
        check(x, L, T=0.8)


# ---- Theorem 2 with dynamic pruning: hs_candidate_mass ----------------------------------------

def _target_lse(xd_target, V, T):
    B, K, ld = xd_target.shape
    _, lse, _ = hs.softmax_stats(xd_target.reshape(B * K, ld), V=V, temperature=T)
    return lse.reshape(B, K)


@pytest.mark.parametrize("dtype", [synth.BF16, synth.F32, synth.F16])
def test_candidate_mass_of_pruned_children(dtype):
    # the children hs_eval_topl returns, then pruned (a seeded mask empties some slots): the
    # unpruned sets give hs_eval_topl's own gamma, the pruned ones the oracle's mass
    w = synth.variant(WL["qwen3_8b_single"], B=2, K=3, N=5, V=20011, ld=20016, dtype=dtype,
                      scales=[0.3 + 0.2 * i for i in range(5)], permute=False)
    note("candidate mass of pruned children dtype=%d" % dtype)
    x = synth.generate(w)
    xd = to_dev(x)
    T, L = 0.8, 10
    out = hs.eval_topl(xd, L=L, V=w.V, temperature=T, want_gamma=True, want_children=True)
    lse = _target_lse(xd[0], w.V, T)
    full = hs.candidate_mass(xd[0], lse, out["children"], V=w.V, temperature=T)
    torch.cuda.synchronize()
    assert np.abs(full.cpu().numpy() - out["gamma"].cpu().numpy()).max() <= GAMMA_TOL
    cand = out["children"].cpu().numpy().copy()
    rng = np.random.default_rng(7)
    cand[rng.random(cand.shape) < 0.4] = -1
    got = hs.candidate_mass(xd[0], lse, torch.from_numpy(cand).cuda(), V=w.V, temperature=T)
    torch.cuda.synchronize()
    ref = oracle.candidate_mass(x[0], cand.transpose(0, 2, 1, 3), V=w.V, T=T)  # [B][K][N]
    assert np.abs(got.cpu().numpy() - ref.transpose(0, 2, 1)).max() <= GAMMA_TOL


@pytest.mark.parametrize("dtype", [synth.BF16, synth.F32, synth.F16])
def test_candidate_mass_long_lists_duplicates_and_bad_indices(dtype):
    # C = 150 slots (three passes of a wave), duplicates counted per listing, empty slots,
    # whole empty sets (mass 0) and one index past V (NaN for that output only)
    w = synth.variant(WL["qwen3_8b_single"], B=3, K=2, N=4, V=3001, ld=3008, dtype=dtype,
                      scales=[0.3 + 0.2 * i for i in range(4)], permute=False)
    note("candidate mass long lists dtype=%d" % dtype)
    x = synth.generate(w)
    xd = to_dev(x)
    rng = np.random.default_rng(8)
    C = 150
    cand = rng.integers(-1, w.V, size=(w.B, w.N, w.K, C)).astype(np.int32)
    cand[0, 1, 0, 5:9] = cand[0, 1, 0, 0]  # duplicates
    cand[1, 2, 1, :] = -1                  # an empty set
    cand[2, 3, 0, 77] = w.V                # past the row end
    for T in (1.0, 0.6):
        lse = _target_lse(xd[0], w.V, T)
        got = hs.candidate_mass(xd[0], lse, torch.from_numpy(cand).cuda(), V=w.V,
                                temperature=T).cpu().numpy()
        ref = oracle.candidate_mass(x[0], cand.transpose(0, 2, 1, 3), V=w.V, T=T).transpose(0, 2, 1)
        nan = np.isnan(ref)
        assert nan.sum() == 1 and nan[2, 3, 0]
        assert np.array_equal(np.isnan(got), nan)
        assert got[1, 2, 1] == 0.0
        assert np.abs(got[~nan] - ref[~nan]).max() <= GAMMA_TOL
