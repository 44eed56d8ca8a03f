"""GPU parity at the edges of the logit range and of the wait protocol.

- Masks: tails and scattered entries at the storage type's most negative finite value (the
  usual masking value) and at -1e9, next to ordinary logits, at several temperatures: every
  masked entry contributes its exact probability, which is 0, so alpha, agreement and the
  argmax match the oracle at the usual bars (hs_eval_alpha through both kernel forms,
  hs_softmax_stats, hs_eval_topl).
- The documented range: rows whose largest logits sit near |z| log2(e) / T = 2^27.
- A NaN logit inside an otherwise -inf run: the row has no distribution, so its normaliser
  and every alpha it takes part in are NaN on both sides.
- The failure path, forced from the host (every bounded wait gives up at once): outputs are
  marked invalid, the learner state stays as it was, and the next call is correct again.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_20064_amd as hs
import synth

pytestmark = pytest.mark.gpu

ALPHA_TOL = 2e-5
W_TOL = 1e-5
BASE = synth.workloads()["qwen3_8b_single"]
F32_MIN = np.float32(np.finfo(np.float32).min)
BF16_MIN = np.uint16(0xFF7F)  # -3.3895e38, the most negative finite bf16


def note(msg):
    print("\n[case] " + msg, flush=True)


def _bf16_bits(a: np.ndarray) -> np.ndarray:
    u = np.asarray(a, np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[np.isnan(a)] = 0x7FC0
    return r


def to_dev(x):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if x.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.cuda()


def logits(B, N, K, V, dtype, seed):
    step = 8 if dtype == synth.BF16 else 4
    w = synth.variant(BASE, B=B, N=N, K=K, V=V, ld=(V + step - 1) // step * step, dtype=dtype,
                      scales=[0.3 + 0.5 * j for j in range(N)], permute=False, seed=seed,
                      nboost=min(20, V // 8))
    return w, synth.generate(w)


def compare_eval(x, V, T):
    out = hs.eval_alpha(to_dev(x), V=V, temperature=T, mode=hs.SAMPLE, want_alpha=True,
                        want_agree=True, want_argmax=True)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.evaluate(x, V=V, T=T, want_alpha=True)
    ra = ref["alpha"].transpose(0, 2, 1)
    assert not np.isnan(ra).any()
    err = np.abs(got["alpha"] - ra).max()
    assert err <= ALPHA_TOL, err
    assert np.array_equal(got["agree"], ref["agree"].transpose(0, 2, 1))
    assert np.array_equal(got["argmax_t"], ref["argmax"][:, :, 0])
    assert np.array_equal(got["argmax_d"], ref["argmax"][:, :, 1:].transpose(0, 2, 1))
    return err


@pytest.mark.parametrize("mask", ["type_min", "minus_1e9"])
@pytest.mark.parametrize("T", [0.5, 1.0, 2.0])
@pytest.mark.parametrize("shape", ["one item per team", "several items per team"])
@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_masked_logits_contribute_nothing(dtype, shape, T, mask):
    if shape == "one item per team":
        B, N, K, V = 1, 5, 3, 20011
    else:
        B, N, K, V = 48, 3, 8, 6151
    note("masks %s at T=%g: %s dtype=%d" % (mask, T, shape, dtype))
    w, x = logits(B, N, K, V, dtype, seed=70 + int(T * 10))
    rng = np.random.default_rng(int(T * 100) + dtype)
    bf = dtype == synth.BF16
    mval = (BF16_MIN if bf else F32_MIN) if mask == "type_min" else (
        _bf16_bits(np.array([-1e9]))[0] if bf else np.float32(-1e9))
    # a padded tail of every row, whole 16-byte vectors and slices of it, and scattered entries
    tail = V - V // 3
    x[:, :, :, tail:V] = mval
    for r in range(w.R):
        for b in range(B):
            for k in range(K):
                x[r, b, k, rng.integers(0, tail, 40)] = mval
    err = compare_eval(x, V, T)
    # the standalone statistics on the same rows
    rows = x.reshape(-1, x.shape[-1])
    mx, lse, am = hs.softmax_stats(to_dev(rows), V=V, temperature=T)
    torch.cuda.synchronize()
    rm, ra, rl = oracle.softmax_stats(rows, V=V, T=T)
    assert np.array_equal(am.cpu().numpy(), ra)
    assert np.allclose(lse.cpu().numpy(), rl, rtol=2e-6, atol=1e-5)
    print("alpha max err %.2e" % err, flush=True)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_masked_logits_topl(dtype):
    note("top-L mass with masked tails, dtype=%d" % dtype)
    w, x = logits(2, 4, 3, 9000, dtype, seed=81)
    bf = dtype == synth.BF16
    x[:, :, :, 6000:9000] = BF16_MIN if bf else F32_MIN
    x[0, 1, 2, 100:3000] = BF16_MIN if bf else F32_MIN
    for T in (0.5, 1.0, 2.0):
        out = hs.eval_topl(to_dev(x), L=10, V=9000, temperature=T, mode=hs.SAMPLE,
                           want_gamma=True, want_hit=True, want_children=True)
        torch.cuda.synchronize()
        ref = oracle.topl(x, 10, V=9000, T=T, want_mass=True)
        g = out["gamma"].cpu().numpy()
        assert np.abs(g - ref["gamma"].transpose(0, 2, 1)).max() <= ALPHA_TOL
        assert np.array_equal(out["children"].cpu().numpy(), ref["idx"].transpose(0, 2, 1, 3))


@pytest.mark.parametrize("shape", ["one item per team", "several items per team"])
def test_logits_near_the_documented_range(shape):
    # fp32 logits around +-9e7 (|z| log2(e) / T about 2^27 at T = 1): the offsets are ~1.3e8
    # with a nudge of about 31 exponent units; every probability keeps fp32 accuracy
    if shape == "one item per team":
        B, N, K, V = 1, 4, 2, 9000
    else:
        B, N, K, V = 40, 2, 8, 4100
    note("logits near 2^27 in scaled units: %s" % shape)
    rng = np.random.default_rng(5)
    R = N + 1
    base = rng.choice([-9.0e7, 9.0e7])
    # distinct fp32 values 8 apart (the spacing of fp32 at 9e7), a handful within a few units
    steps = rng.integers(-6, 2, (R, B, K, V)).astype(np.float64)
    x = (base + 8.0 * steps).astype(np.float32)
    assert np.all(np.abs(x.astype(np.float64) - (base + 8.0 * steps)) == 0)
    compare_eval(x, V, 1.0)
    compare_eval(x, V, 16.0)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_nan_inside_a_minus_inf_run(dtype):
    # a row whose first logits are -inf with a NaN among them, finite logits after: no
    # distribution (NaN normaliser, NaN alpha for the pairs it is in)
    note("NaN inside a -inf run, dtype=%d" % dtype)
    B, N, K, V = 2, 3, 2, 12000
    w, x = logits(B, N, K, V, dtype, seed=91)
    bf = dtype == synth.BF16
    ninf = np.uint16(0xFF80) if bf else np.float32(-np.inf)
    nan = np.uint16(0x7FC0) if bf else np.float32(np.nan)
    x[2, 1, 0, :5000] = ninf  # drafter 1 at (b=1, k=0)
    x[2, 1, 0, 1234] = nan
    x[0, 0, 1, :3000] = ninf  # the target at (b=0, k=1)
    x[0, 0, 1, 17] = nan
    out = hs.eval_alpha(to_dev(x), V=V, temperature=1.0, mode=hs.SAMPLE, want_alpha=True)
    torch.cuda.synchronize()
    got = out["alpha"].cpu().numpy()
    ref = oracle.evaluate(x, V=V, T=1.0, want_alpha=True)["alpha"].transpose(0, 2, 1)
    want_nan = np.zeros((B, N, K), bool)
    want_nan[1, 1, 0] = True
    want_nan[0, :, 1] = True
    assert np.array_equal(np.isnan(ref), want_nan)
    assert np.array_equal(np.isnan(got), want_nan)
    assert np.abs(got[~want_nan] - ref[~want_nan]).max() <= ALPHA_TOL
    rows = x.reshape(-1, x.shape[-1])
    _, lse, _ = hs.softmax_stats(to_dev(rows), V=V, temperature=1.0)
    torch.cuda.synchronize()
    _, _, rl = oracle.softmax_stats(rows, V=V, T=1.0)
    assert np.array_equal(np.isnan(lse.cpu().numpy()), np.isnan(rl))
    assert np.isnan(rl).sum() == 2


@pytest.mark.parametrize("mode", [hs.SAMPLE, hs.GREEDY])
def test_failed_round_leaves_learner_state_unchanged(mode):
    # every bounded wait gives up at once (forced from the host): the call's outputs are marked
    # invalid, no learner consumes the lost words, and the following call is exact again
    note("forced failure path, mode=%d" % mode)
    w = synth.variant(BASE, B=3, N=8, K=4, V=40000, mode=mode)
    x = synth.generate(w)
    xd = to_dev(x)
    rnd = hs.Round(xd, V=w.V, temperature=1.0, mode=mode, loss_kind=w.loss, eta=w.eta)
    rnd.run()  # a first good round moves the state away from uniform
    torch.cuda.synchronize()
    st = rnd.state
    before = {k: getattr(st, k).clone() for k in ("logw", "w", "R", "p", "c")}
    try:
        hs.set_wait_limit(0)
        rnd.run()
        torch.cuda.synchronize()
    finally:
        hs.set_wait_limit(-1)
    for k, v in before.items():
        assert torch.equal(getattr(st, k), v), k
    assert torch.isnan(rnd.eal).all()
    if mode == hs.SAMPLE:
        assert torch.isnan(rnd.alpha).all()
    else:
        assert int(rnd.agree.sum()) == 0
    # the next call uses a new tag and is exact again
    rnd.run()
    torch.cuda.synchronize()
    ref = oracle.evaluate(x, V=w.V, T=1.0, want_alpha=(mode == hs.SAMPLE))
    gam = (ref["alpha"] if mode == hs.SAMPLE else ref["agree"].astype(np.float64))
    gam = gam.transpose(0, 2, 1)
    acc = oracle.accept_len(gam, loss_kind=w.loss)
    w_or = np.full((w.B, w.N), 1.0 / w.N)
    R_or = np.zeros((w.B, w.N))
    p_or = np.full((w.B, w.N), 1.0 / w.N)
    for _ in range(2):  # two good rounds of the same logits on the oracle side
        w_or = oracle.hedge(w_or, acc["loss"], w.eta)
        R_or, p_or, _ = oracle.normalhedge(R_or, p_or, acc["loss"])
    eal = rnd.eal.cpu().numpy()
    assert np.all(np.abs(eal - acc["eal"]) <= 1e-4 * acc["eal"])
    assert np.abs(st.w.cpu().numpy() - w_or).max() <= W_TOL
    assert np.abs(st.p.cpu().numpy() - p_or).max() <= W_TOL
