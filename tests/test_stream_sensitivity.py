"""How much NormalHedge amplifies fp32-level perturbations of alpha over a long stream.

This fixes the end-to-end bound used for the 1000-round stream parity test. The oracle
pipeline (alpha -> Theorem 3 EAL -> length loss -> NormalHedge) is run twice on the same
seeded logits of the large-pool workload (B=32, N=64, K=8, regime switch at round 500) at
V=64: once exactly, once with every alpha multiplied by (1 + 2e-7 * Z), the size of fp32
arithmetic error. The distributions separate by more than the 1e-5 weight tolerance, so no
fp32 evaluation of alpha could hold 1e-5 end to end; they stay well below 3e-4.
"""
import numpy as np

import oracle
import synth


def test_normalhedge_amplifies_fp32_level_alpha_noise():
    w = synth.variant(synth.workloads()["large_pool_stream"], V=64)
    B, N = w.B, w.N
    rng = np.random.default_rng(0)
    R0, p0 = np.zeros((B, N)), np.full((B, N), 1 / N)
    R1, p1 = R0.copy(), p0.copy()
    w0, w1 = p0.copy(), p0.copy()
    dp = dw = 0.0
    for r in range(1000):
        x = synth.generate(w, round=r)
        a = oracle.evaluate(x, T=1.0)["alpha"].transpose(0, 2, 1)
        l0 = oracle.accept_len(a, loss_kind=w.loss)["loss"]
        l1 = oracle.accept_len(a * (1 + rng.normal(0, 2e-7, a.shape)), loss_kind=w.loss)["loss"]
        R0, p0, _ = oracle.normalhedge(R0, p0, l0)
        R1, p1, _ = oracle.normalhedge(R1, p1, l1)
        w0 = oracle.hedge(w0, l0, w.eta)
        w1 = oracle.hedge(w1, l1, w.eta)
        dp = max(dp, np.abs(p0 - p1).max())
        dw = max(dw, np.abs(w0 - w1).max())
    assert 1e-5 < dp < 3e-4, dp
    assert dw < 1e-5, dw
