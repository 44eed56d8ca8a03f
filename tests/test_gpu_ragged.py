"""GPU parity for chunks of ragged verified length k_h (Appendix "Chunk-Level vs Token-Level"):
a chain's path_end[b] = k_h - 1 per query. EAL and the losses against the oracle on the same
gamma (fp64 on both sides: 1e-12), the round's alpha within 2e-5, the learners within 1e-5."""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_20064_amd as hs
import synth

pytestmark = pytest.mark.gpu


def note(msg):
    print("\n[case] " + msg, flush=True)


@pytest.mark.parametrize("loss_kind", [hs.LOSS_LENGTH, hs.LOSS_ACCEPT_CHUNK, hs.LOSS_ACCEPT_TOKEN])
def test_accept_len_ragged_chunks(loss_kind):
    rng = np.random.default_rng(41)
    B, N, K = 6, 5, 8
    g = rng.random((B, N, K)).astype(np.float32)
    ends = np.array([0, 7, 3, 5, 1, 6], dtype=np.int32)
    note("accept_len ragged loss=%d" % loss_kind)
    out = hs.accept_len(torch.from_numpy(g).cuda(), mode=hs.SAMPLE,
                        path_end=torch.from_numpy(ends).cuda(), loss_kind=loss_kind)
    torch.cuda.synchronize()
    ref = oracle.accept_len(g.astype(np.float64), path_end=ends, loss_kind=loss_kind)
    assert np.allclose(out["eal"].cpu().numpy(), ref["eal"], rtol=1e-12, atol=0)
    assert np.allclose(out["loss"].cpu().numpy(), ref["loss"], rtol=0, atol=1e-12)
    if loss_kind == hs.LOSS_ACCEPT_TOKEN:
        lo = out["loss"].cpu().numpy()
        for b, e in enumerate(ends):
            assert np.all(lo[e + 1:, b] == 0.0)


@pytest.mark.parametrize("loss_kind", [hs.LOSS_LENGTH, hs.LOSS_ACCEPT_TOKEN])
def test_round_with_ragged_chunks(loss_kind):
    w = synth.variant(synth.workloads()["qwen3_8b_single"], B=4, V=20000, loss=loss_kind)
    x = synth.generate(w)
    ends = np.array([7, 2, 0, 4], dtype=np.int32)
    note("round ragged loss=%d" % loss_kind)
    xd = torch.from_numpy(x).view(torch.bfloat16).cuda()
    rnd = hs.Round(xd, V=w.V, temperature=w.temperature, mode=hs.SAMPLE, loss_kind=loss_kind,
                   eta=w.eta, path_end=torch.from_numpy(ends).cuda())
    rnd.run()
    torch.cuda.synchronize()
    alpha = rnd.alpha.cpu().numpy().astype(np.float64)
    ref = oracle.evaluate(x, V=w.V, T=w.temperature)["alpha"].transpose(0, 2, 1)
    assert np.abs(alpha - ref).max() <= 2e-5
    acc = oracle.accept_len(alpha, path_end=ends, loss_kind=loss_kind)  # same-input check
    assert np.allclose(rnd.eal.cpu().numpy(), acc["eal"], rtol=1e-12, atol=0)
    w_or = oracle.hedge(np.full((w.B, w.N), 1.0 / w.N), acc["loss"], w.eta)
    _, p_or, _ = oracle.normalhedge(np.zeros((w.B, w.N)), np.full((w.B, w.N), 1.0 / w.N), acc["loss"])
    assert np.abs(rnd.state.w.cpu().numpy() - w_or).max() <= 1e-5
    assert np.abs(rnd.state.p.cpu().numpy() - p_or).max() <= 1e-5
