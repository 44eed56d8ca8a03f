"""GPU parity over a seeded sweep of shapes: hs_eval_alpha and hs_eval_topl against the oracle.

Each case draws B, N, K, V, the dtype, the temperature and the mode from its seed, so that
together the cases cross the launch geometry's edges:
- one and several row sets per group (N up to 20, sets of at most 8 drafters);
- one and several slices per row, with ragged tails (V not a multiple of the 2048-logit slice
  or of the 16-byte vector);
- teams that hold one item and teams that run several;
- drafter rows at a constant distance and rows in separate allocations (the row table).
Tolerances as in the other parity tests: indices bit-exact, alpha and gamma within 2e-5.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_20064_amd as hs
import synth

pytestmark = pytest.mark.gpu

ALPHA_TOL = 2e-5
BASE = synth.workloads()["qwen3_8b_single"]


def _bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even bf16 bit patterns of fp32 values (NaN stays a NaN pattern)."""
    u = np.asarray(a, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[np.isnan(a)] = 0x7FC0
    return r


def note(msg):
    print("\n[case] " + msg, flush=True)


def draw(seed):
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, 5))
    N = int(rng.integers(1, 21))
    K = int(rng.integers(1, 6))
    V = int(rng.choice([1, 7, 2048, 2049, 4095, int(rng.integers(8, 30000))]))
    dtype = int(rng.choice([synth.F32, synth.BF16]))
    step = 8 if dtype == synth.BF16 else 4  # 16-byte row starts
    ld = (V + step - 1) // step * step + step * int(rng.integers(0, 2))
    T = float(rng.choice([0.4, 1.0, 3.0]))
    mode = int(rng.choice([hs.SAMPLE, hs.GREEDY]))
    scattered = bool(seed % 3 == 2)
    w = synth.variant(BASE, B=B, N=N, K=K, V=V, ld=ld, dtype=dtype,
                      scales=[0.2 + 0.3 * i for i in range(N)], permute=True, seed=seed,
                      nboost=min(BASE.nboost, V // 4))
    return w, T, mode, scattered


def to_dev(w, x):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if w.dtype == synth.BF16:
        t = t.view(torch.bfloat16)
    return t.cuda()


def split(xd, scattered):
    """The target and the list of drafter tensors; when scattered, each drafter is a copy in
    an allocation of its own, with allocations of uneven size between them."""
    if not scattered:
        return xd[0], list(xd[1:])
    keep, ds = [], []
    for i in range(1, xd.shape[0]):
        keep.append(torch.empty(4096 + 53 * i, dtype=torch.uint8, device="cuda"))
        ds.append(xd[i].clone())
    return xd[0], ds


# Many row sets over few slices, so that each team runs several items (the pipelined kernel
# with dynamically claimed row sets): (B, N, K, V, dtype, mode, scattered).
MANY = [(64, 12, 6, 4099, synth.BF16, hs.SAMPLE, False),
        (64, 5, 8, 2056, synth.F32, hs.GREEDY, True),
        (40, 9, 4, 6001, synth.BF16, hs.SAMPLE, True)]


def many(i):
    B, N, K, V, dtype, mode, scattered = MANY[i]
    step = 8 if dtype == synth.BF16 else 4
    w = synth.variant(BASE, B=B, N=N, K=K, V=V, ld=(V + step - 1) // step * step, dtype=dtype,
                      scales=[0.2 + 0.3 * j for j in range(N)], permute=True, seed=50 + i)
    return w, 0.8, mode, scattered


@pytest.mark.parametrize("seed", range(16 + len(MANY)))
def test_eval_alpha_sweep(seed):
    w, T, mode, scattered = draw(seed) if seed < 16 else many(seed - 16)
    note("alpha seed=%d B=%d N=%d K=%d V=%d ld=%d dtype=%d T=%g mode=%d scattered=%d"
         % (seed, w.B, w.N, w.K, w.V, w.row_ld, w.dtype, T, mode, scattered))
    x = synth.generate(w)
    t, ds = split(to_dev(w, x), scattered)
    out = hs.eval_alpha(t, ds, V=w.V, temperature=T, mode=mode, want_alpha=(mode == hs.SAMPLE),
                        want_agree=True, want_argmax=True)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.evaluate(x, V=w.V, T=T, want_alpha=(mode == hs.SAMPLE))
    if mode == hs.SAMPLE:
        err = np.abs(got["alpha"] - ref["alpha"].transpose(0, 2, 1)).max()
        assert err <= ALPHA_TOL, err
    assert np.array_equal(got["agree"], ref["agree"].transpose(0, 2, 1))
    assert np.array_equal(got["argmax_t"], ref["argmax"][:, :, 0])
    assert np.array_equal(got["argmax_d"], ref["argmax"][:, :, 1:].transpose(0, 2, 1))


@pytest.mark.parametrize("seed", range(8))
def test_eval_topl_sweep(seed):
    w, T, mode, _ = draw(100 + seed)
    L = int(np.random.default_rng(seed).integers(1, min(w.V, hs.MAX_TOPL) + 1))
    note("topl seed=%d B=%d N=%d K=%d V=%d ld=%d dtype=%d T=%g mode=%d L=%d"
         % (seed, w.B, w.N, w.K, w.V, w.row_ld, w.dtype, T, mode, L))
    x = synth.generate(w)
    out = hs.eval_topl(to_dev(w, x), L=L, V=w.V, temperature=T, mode=mode,
                       want_gamma=(mode == hs.SAMPLE), want_hit=True, want_children=True)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.topl(x.reshape(x.shape[0], w.B * w.K, -1), L, V=w.V, T=T,
                      want_mass=(mode == hs.SAMPLE))
    for b in range(w.B):
        for k in range(w.K):
            g = b * w.K + k
            assert np.array_equal(got["children"][b, :, k], ref["idx"][g]), (b, k)
            assert np.array_equal(got["hit"][b, :, k], ref["hit"][g]), (b, k)
            if mode == hs.SAMPLE:
                assert np.abs(got["gamma"][b, :, k] - ref["gamma"][g]).max() <= ALPHA_TOL, (b, k)


# The largest rows the evaluation takes (512 slices: V = 2^20 bf16, 2^19 fp32): one item per
# team, and one team of 512 workgroups running several items with claimed row sets.
LIMIT = [(1, 3, 1, 1 << 20, synth.BF16, hs.SAMPLE),
         (2, 3, 2, 1 << 20, synth.BF16, hs.SAMPLE),
         (1, 9, 2, 1 << 19, synth.F32, hs.GREEDY)]


@pytest.mark.parametrize("case", range(len(LIMIT)))
def test_eval_alpha_at_the_vocabulary_limit(case):
    B, N, K, V, dtype, mode = LIMIT[case]
    note("alpha at the limit B=%d N=%d K=%d V=%d dtype=%d mode=%d" % (B, N, K, V, dtype, mode))
    w = synth.variant(BASE, B=B, N=N, K=K, V=V, ld=V, dtype=dtype,
                      scales=[0.2 + 0.3 * j for j in range(N)], permute=False, seed=70 + case)
    x = synth.generate(w)
    xd = to_dev(w, x)
    out = hs.eval_alpha(xd[0], list(xd[1:]), V=V, temperature=1.0, mode=mode,
                        want_alpha=(mode == hs.SAMPLE), want_agree=True, want_argmax=True)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.evaluate(x, V=V, T=1.0, want_alpha=(mode == hs.SAMPLE))
    if mode == hs.SAMPLE:
        assert np.abs(got["alpha"] - ref["alpha"].transpose(0, 2, 1)).max() <= ALPHA_TOL
    assert np.array_equal(got["agree"], ref["agree"].transpose(0, 2, 1))
    assert np.array_equal(got["argmax_t"], ref["argmax"][:, :, 0])
    assert np.array_equal(got["argmax_d"], ref["argmax"][:, :, 1:].transpose(0, 2, 1))


def _dead_rows_case(B, N, K, V, dtype, dead, nan_logit=False):
    """Logits with whole rows at -inf (or, nan_logit, one NaN logit in each such row plus a
    large logit elsewhere): dead = list of (row, b, k), row 0 the target."""
    step = 4 if dtype == synth.F32 else 8
    w = synth.variant(BASE, B=B, N=N, K=K, V=V, ld=(V + step - 1) // step * step, dtype=dtype,
                      scales=[0.3 + 0.4 * j for j in range(N)], permute=False, seed=90)
    x = synth.generate(w)
    bf = dtype == synth.BF16
    ft = np.float16 if dtype == synth.F16 else np.float32
    for j, (r, b, k) in enumerate(dead):
        if nan_logit:
            x[r, b, k, (37 * j + 11) % V] = np.uint16(0x7FC0) if bf else ft(np.nan)
            x[r, b, k, (53 * j + 5) % V] = np.uint16(0x4248) if bf else ft(50.0)
        else:
            x[r, b, k, :V] = np.uint16(0xFF80) if bf else ft(-np.inf)
    return w, x


@pytest.mark.parametrize("nan_logit", [False, True])
@pytest.mark.parametrize("shape", ["one item per team", "several items per team"])
@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16, synth.F16])
def test_alpha_is_nan_where_a_row_has_no_distribution(shape, dtype, nan_logit):
    # Theorem 1 needs two distributions: a row of -inf logits has none, and neither has a row
    # holding a NaN logit. Alpha is NaN for every drafter when the target's row is such a row
    # and for that drafter alone otherwise; agreement and argmax keep their rule (lowest index
    # of the max, a NaN never being larger).
    if shape == "one item per team":
        B, N, K, V = 1, 3, 3, 5000
        dead = [(0, 0, 0), (2, 0, 1)]
    else:
        B, N, K, V = 64, 3, 8, 2056
        dead = [(0, 5, 3), (1, 17, 0), (3, 40, 7), (0, 63, 7), (2, 63, 7)]
    note("dead rows: %s dtype=%d nan_logit=%d" % (shape, dtype, nan_logit))
    w, x = _dead_rows_case(B, N, K, V, dtype, dead, nan_logit)
    out = hs.eval_alpha(to_dev(w, x)[0], list(to_dev(w, x)[1:]), V=V, temperature=1.0,
                        mode=hs.SAMPLE, want_alpha=True, want_agree=True, want_argmax=True)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.evaluate(x, V=V, T=1.0, want_alpha=True)
    ra = ref["alpha"].transpose(0, 2, 1)
    nan = np.isnan(ra)
    want = np.zeros((B, N, K), bool)  # [B][N][K]: the pairs with a dead row
    for r, b, k in dead:
        if r == 0:
            want[b, :, k] = True
        else:
            want[b, r - 1, k] = True
    assert np.array_equal(nan, want)
    assert np.array_equal(np.isnan(got["alpha"]), nan)
    assert np.abs(got["alpha"][~nan] - ra[~nan]).max() <= ALPHA_TOL
    assert np.array_equal(got["agree"], ref["agree"].transpose(0, 2, 1))
    assert np.array_equal(got["argmax_t"], ref["argmax"][:, :, 0])
    assert np.array_equal(got["argmax_d"], ref["argmax"][:, :, 1:].transpose(0, 2, 1))


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16, synth.F16])
def test_softmax_stats_of_rows_without_a_distribution(dtype):
    # hs_softmax_stats on rows of -inf and rows holding a NaN: the normaliser is NaN, the max
    # and argmax skip the NaN (an all -inf row has max -inf at index 0); the other rows as usual
    note("softmax stats, dead and NaN rows, dtype=%d" % dtype)
    V, rows = 9001, 6
    ld = (V + 7) // 8 * 8
    rng = np.random.default_rng(5)
    z = rng.normal(0, 2, (rows, ld)).astype(np.float32)
    z[:, V:] = 0.0
    z[1, :V] = -np.inf
    z[3, 4000] = np.nan
    z[3, 77] = 30.0
    z[4, [0, 8999]] = np.nan
    x = _bf16_bits(z) if dtype == synth.BF16 else z.astype(np.float16) if dtype == synth.F16 else z
    t = torch.from_numpy(x)
    t = (t.view(torch.bfloat16) if dtype == synth.BF16 else t).cuda()
    for T in (1.0, 0.6):
        mx, lse, am = hs.softmax_stats(t, V=V, temperature=T)
        torch.cuda.synchronize()
        rm, ra, rl = oracle.softmax_stats(x, V=V, T=T)
        assert np.array_equal(am.cpu().numpy(), ra)
        assert np.array_equal(mx.cpu().numpy().astype(np.float64), rm)
        got = lse.cpu().numpy()
        assert np.array_equal(np.isnan(got), np.isnan(rl)) and np.isnan(rl[[1, 3, 4]]).all()
        ok = ~np.isnan(rl)
        assert np.allclose(got[ok], rl[ok], rtol=2e-6, atol=1e-5)
