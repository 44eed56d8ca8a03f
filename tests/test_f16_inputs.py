"""fp16 logits (IEEE binary16, the precision the paper's models were served in: Section
"Experiment setup and baselines"): pins of the oracle's decoding and of the generator's
rounding against numpy's own binary16 type, which shares no code with either.

The oracle reads every stored type through one decode step, so decoding every fp16 bit
pattern exactly, and giving the same alpha, argmax, Top_L and statistics as for the same
values stored as fp32, ties its fp16 path to the already pinned fp32 one.
"""
import numpy as np
import pytest

import oracle
import synth


def test_oracle_decodes_every_fp16_pattern_exactly():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = bits.view(np.float16).reshape(-1, 1)  # one single-logit row per pattern
    m, a, l = oracle.softmax_stats(x, T=1.0)
    ref = x[:, 0].astype(np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(m[fin], ref[fin])
    # a one-logit row: log sum exp(z) = z exactly
    assert np.array_equal(l[fin], ref[fin])
    assert np.all(a == 0)
    # +inf is the maximum of its row; -inf leaves a row with no distribution (lse NaN)
    pinf = ref == np.inf
    assert np.all(m[pinf] == np.inf)
    ninf = ref == -np.inf
    assert np.all(np.isnan(l[ninf]))
    # NaN patterns: the row's statistics are not finite
    nan = np.isnan(ref)
    assert nan.sum() == 2 * 1023
    assert not np.any(np.isfinite(l[nan]))


@pytest.mark.parametrize("seed", [0, 1])
def test_generator_rounds_like_ieee_binary16(seed):
    rng = np.random.default_rng(seed)
    xs = list(rng.normal(0.0, 1.0, 2000) * 10.0 ** rng.uniform(-9, 5, 2000))
    # the edges: the largest finite value, the overflow threshold (65520 rounds to infinity,
    # just below it to 65504), the subnormal range and its ties, signed zeros, infinities
    xs += [65504.0, 65519.99, 65520.0, 65536.0, 1e6, 2.0 ** -14, 2.0 ** -24, 2.0 ** -25,
           3 * 2.0 ** -26, 2.0 ** -25 * 1.0000001, 5 * 2.0 ** -26, 2.0 ** -14 - 2.0 ** -25,
           2.0 ** -14 - 2.0 ** -26, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, 0.0, -0.0,
           np.inf, -np.inf, 1e-40, -1e-40]
    xs += [-v for v in xs[-22:-5]]
    for x in xs:
        got = synth.round_f16(x)
        with np.errstate(over="ignore"):
            f = np.array([x], dtype=np.float32).astype(np.float16)
        want = int(f.view(np.uint16)[0])
        assert got == want, (x, hex(got), hex(want))
    assert np.isnan(np.array([synth.round_f16(float("nan"))], dtype=np.uint16).view(np.float16)[0])


def _f16_workload():
    w = synth.workloads()["tiny_chain"]
    return synth.Workload(**{**w.__dict__, "dtype": synth.F16, "V": 3001, "N": 3, "K": 3,
                             "scales": w.scales[:3]})


def test_generated_fp16_logits_are_rounded_fp32_ones():
    w = _f16_workload()
    x16 = synth.generate(w)
    assert x16.dtype == np.float16 and np.all(np.isfinite(x16))
    t32 = synth.generate(synth.Workload(**{**w.__dict__, "dtype": synth.F32}), rows=[0])
    # the target row is the same draw rounded to binary16 instead of fp32
    assert np.array_equal(x16[0], t32[0].astype(np.float16))
    assert synth.decode(w, x16).dtype == np.float64


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_oracle_fp16_path_equals_its_fp32_path_on_the_same_values(T):
    w = _f16_workload()
    x16 = synth.generate(w)
    # ties and specials of the fp16 grid: a repeated maximum, -0 against +0, -inf entries
    x16[1, 0, 0, 5] = x16[1, 0, 0].max()
    x16[1, 0, 0, 9] = x16[1, 0, 0, 5]
    x16[2, 0, 1, 3] = np.float16(-0.0)
    x16[0, 0, 2, 17] = np.float16(-np.inf)
    x32 = x16.astype(np.float32)  # every binary16 value is an fp32 value
    e16, e32 = oracle.evaluate(x16, T=T), oracle.evaluate(x32, T=T)
    for k in ("alpha", "agree", "argmax", "rmax", "rlse"):
        assert np.array_equal(e16[k], e32[k]), k
    t16, t32 = oracle.topl(x16, 10, T=T), oracle.topl(x32, 10, T=T)
    for k in ("gamma", "hit", "idx"):
        assert np.array_equal(t16[k], t32[k]), k
    rows16, rows32 = x16.reshape(-1, w.V), x32.reshape(-1, w.V)
    for a, b in zip(oracle.softmax_stats(rows16, T=T), oracle.softmax_stats(rows32, T=T)):
        assert np.array_equal(a, b)
