"""hs_eval_alpha_noalloc (the fixed device workspace) against hs_eval_alpha (a workspace of the
caller's), through the C ABI: calls in a row, each on a smaller input than the last, each compared
with hs_eval_alpha on the same logits at the parity bars (indices and agreement bit-exact, alpha
within 2e-5; the two share their kernels, so alpha agrees bit for bit as well)."""
import numpy as np
import pytest
import torch

import paper_2510_20064_amd as hs
import synth

pytestmark = pytest.mark.gpu

BASE = synth.workloads()["qwen3_8b_single"]


def _dev(x):
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.view(torch.bfloat16).cuda() if x.dtype == np.uint16 else t.cuda()


def _outs(B, N, K):
    return {"alpha": torch.empty((B, N, K), dtype=torch.float32, device="cuda"),
            "agree": torch.empty((B, N, K), dtype=torch.uint8, device="cuda"),
            "argmax_t": torch.empty((B, K), dtype=torch.int32, device="cuda"),
            "argmax_d": torch.empty((B, N, K), dtype=torch.int32, device="cuda")}


@pytest.mark.parametrize("mode", [hs.SAMPLE, hs.GREEDY])
def test_noalloc_matches_eval_alpha_on_calls_in_a_row(mode):
    # each call smaller than the one before; the first has groups enough for the teams to take
    # a (query, position)'s two row sets in turn
    shapes = [dict(B=16, N=16, K=8, V=151936), dict(B=3, N=12, K=5, V=151936),
              dict(B=1, N=4, K=2, V=40000)]
    for i, sh in enumerate(shapes):
        print("\n[case] noalloc call %d mode=%d %s" % (i, mode, sh), flush=True)
        w = synth.variant(BASE, scales=[0.2 + 0.3 * j for j in range(sh["N"])], seed=40 + i,
                          permute=False, **sh)
        x = _dev(synth.generate(w))
        B, N, K = w.B, w.N, w.K
        got = _outs(B, N, K)
        hs.eval_alpha_noalloc(x, V=w.V, temperature=0.8, mode=mode, out=got)
        ref = hs.eval_alpha(x, V=w.V, temperature=0.8, mode=mode, want_alpha=True,
                            want_agree=True, want_argmax=True)
        torch.cuda.synchronize()
        a, r = got["alpha"].cpu().numpy(), ref["alpha"].cpu().numpy()
        assert not np.isnan(a).any()
        assert np.abs(a - r).max() <= 2e-5
        assert np.array_equal(a.view(np.uint32), r.view(np.uint32))
        for k in ("agree", "argmax_t", "argmax_d"):
            assert torch.equal(got[k], ref[k]), k
