"""The C ABI on the host: the library loads, exports every declared symbol, and rejects
invalid arguments before any HIP call (so these run without a GPU)."""
import ctypes
import os
import re

import pytest

import paper_2510_20064_amd as hs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hedgespec.h")

FAKE = 0x100000  # never dereferenced: validation fails before any device access


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hs_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = hs.load_library()
    names = declared_functions()
    assert "hs_eval_alpha" in names and "hs_round" in names and len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    lib = hs.load_library()
    assert lib.hs_status_string(0) == b"HS_OK"
    assert lib.hs_status_string(6) == b"HS_ERR_TREE"
    assert lib.hs_status_string(99) == b"HS_ERR_UNKNOWN"
    assert lib.hs_version() >= 100


def test_workspace_size_query():
    lib = hs.load_library()
    assert lib.hs_eval_alpha_workspace_size(1, 8, 8, 151936, 1) > 0
    assert lib.hs_eval_alpha_workspace_size(0, 8, 8, 151936, 1) == 0
    assert lib.hs_eval_alpha_workspace_size(1, 65, 8, 151936, 1) == 0
    assert lib.hs_eval_alpha_workspace_size(1, 8, 8, 151936, 7) == 0


def _views(n, ptr=FAKE, sb=8 * 151936, sk=151936):
    return (hs.hs_view * n)(*[hs.hs_view(ptr + 0x1000000 * (i + 1), sb, sk) for i in range(n)])


def _eval(lib, **kw):
    a = dict(target=hs.hs_view(FAKE, 8 * 151936, 151936), N=8, B=1, K=8, V=151936, dtype=1,
             T=1.0, mode=0, alpha=FAKE, agree=None, argmax_t=None, argmax_d=None, ws=FAKE * 16,
             ws_bytes=1 << 30)
    a.update(kw)
    d = kw.get("drafters", _views(a["N"]))
    tv = a["target"]
    return lib.hs_eval_alpha(ctypes.byref(tv) if tv is not None else None, d, a["N"], a["B"],
                             a["K"], a["V"], a["dtype"], a["T"], a["mode"], a["alpha"], a["agree"],
                             a["argmax_t"], a["argmax_d"], a["ws"], a["ws_bytes"], None)


def test_eval_alpha_validation_codes():
    lib = hs.load_library()
    assert _eval(lib, N=0) == 2
    assert _eval(lib, B=0) == 2
    assert _eval(lib, N=65, drafters=_views(65)) == 8
    assert _eval(lib, K=65) == 8
    assert _eval(lib, dtype=5) == 3
    assert _eval(lib, mode=3) == 10
    assert _eval(lib, target=None) == 1
    assert _eval(lib, alpha=None) == 1  # sample mode needs alpha
    assert _eval(lib, mode=1, alpha=None, agree=None) == 1
    assert _eval(lib, T=0.0) == 5
    assert _eval(lib, T=float("nan")) == 5
    assert _eval(lib, T=-1.0) == 5
    assert _eval(lib, target=hs.hs_view(FAKE + 2, 8 * 151936, 151936)) == 4
    assert _eval(lib, target=hs.hs_view(FAKE, 8 * 151936, 151937)) == 4
    assert _eval(lib, drafters=_views(8, sk=3)) == 4
    assert _eval(lib, ws=None) == 7
    assert _eval(lib, ws_bytes=16) == 7
    assert _eval(lib, ws=FAKE * 16 + 8) == 4
    bad = _views(8)
    bad[3] = hs.hs_view(None, 0, 0)
    assert _eval(lib, drafters=bad) == 1
    assert b"drafter 3" in lib.hs_last_error()
    # 512 slices of 256 16-byte vectors per row at most: V = 2^20 bf16 or 2^19 fp32
    assert _eval(lib, V=(1 << 20) + 1) == 8
    assert _eval(lib, V=(1 << 19) + 1, dtype=0) == 8


def test_accept_len_validation_codes():
    lib = hs.load_library()

    def call(parent=None, mode=0, loss_kind=0, alpha=FAKE, agree=None, eal=FAKE, K=4, N=4):
        arr = None if parent is None else (ctypes.c_int32 * len(parent))(*parent)
        return lib.hs_accept_len(alpha, agree, mode, 2, N, K, arr, None, eal, None, loss_kind,
                                 None, None)

    assert call(parent=[0, 0, 1, 2]) == 6
    assert call(parent=[-1, 1, 1, 2]) == 6
    assert call(parent=[-1, 0, 3, 2]) == 6
    assert call(parent=[-1, 0, 0, 1], loss_kind=1) == 6
    assert call(loss_kind=7) == 10
    assert call(eal=None) == 1
    assert call(mode=1) == 1  # greedy needs agree
    assert call(N=0) == 2
    assert call(K=65) == 8


def test_learner_validation_codes():
    lib = hs.load_library()
    assert lib.hs_hedge_update(None, FAKE, FAKE, 1, 2, 3, 0.5, None) == 1
    assert lib.hs_hedge_update(FAKE, FAKE, FAKE, 0, 2, 3, 0.5, None) == 2
    assert lib.hs_hedge_update(FAKE, FAKE, FAKE, 1, 2, 65, 0.5, None) == 8
    assert lib.hs_hedge_update(FAKE, FAKE, FAKE, 1, 2, 3, float("inf"), None) == 10
    assert lib.hs_normalhedge_update(FAKE, FAKE, None, FAKE, 1, 2, 3, None) == 1
    assert lib.hs_normalhedge_update(FAKE, FAKE, FAKE, FAKE, 1, 0, 3, None) == 2


def test_softmax_stats_validation_codes():
    lib = hs.load_library()
    assert lib.hs_softmax_stats(None, 0, 4, 100, 100, 1.0, FAKE, None, None, None) == 1
    assert lib.hs_softmax_stats(FAKE, 4, 4, 100, 100, 1.0, FAKE, None, None, None) == 3
    assert lib.hs_softmax_stats(FAKE, 0, 4, 100, 99, 1.0, FAKE, None, None, None) == 2
    assert lib.hs_softmax_stats(FAKE, 0, 4, 100, 101, 1.0, FAKE, None, None, None) == 4
    assert lib.hs_softmax_stats(FAKE, 0, 4, 100, 100, 0.0, FAKE, None, None, None) == 5


def test_stream_read_validation_codes():
    lib = hs.load_library()
    assert lib.hs_stream_read(None, 1024, 64, 4, 0, FAKE, None) == 1
    assert lib.hs_stream_read(FAKE, 1024, 64, 4, 0, None, None) == 1
    assert lib.hs_stream_read(FAKE + 8, 1024, 64, 4, 0, FAKE, None) == 4
    assert lib.hs_stream_read(FAKE, 1000, 64, 4, 0, FAKE, None) == 4
    assert lib.hs_stream_read(FAKE, 0, 64, 4, 0, FAKE, None) == 2
    assert lib.hs_stream_read(FAKE, 1024, 0, 4, 0, FAKE, None) == 2
    assert lib.hs_stream_read(FAKE, 1024, 64, 3, 0, FAKE, None) == 10


def test_softmax_stats_binding_rejects_mismatched_outputs():
    # checked before the library is called, so host tensors do
    import torch

    x = torch.zeros((3, 64), dtype=torch.float32)
    bad = [(torch.empty(3), torch.empty(3), torch.empty(3)),                         # argmax f32
           (torch.empty(4), torch.empty(3), torch.empty(3, dtype=torch.int32)),      # wrong length
           (torch.empty(6)[::2], torch.empty(3), torch.empty(3, dtype=torch.int32))]  # strided
    for out in bad:
        with pytest.raises(ValueError):
            hs.softmax_stats(x, out=out)


def test_round_validation_codes():
    lib = hs.load_library()
    d = _views(8)
    a = hs.hs_round_args()
    a.target = hs.hs_view(FAKE, 8 * 151936, 151936)
    a.drafters_host = ctypes.cast(d, ctypes.POINTER(hs.hs_view))
    a.N, a.B, a.K, a.V, a.dtype, a.temperature, a.mode = 8, 1, 8, 151936, 1, 1.0, 0
    a.alpha, a.eal, a.workspace, a.workspace_bytes = FAKE, FAKE, FAKE * 16, 1 << 30
    a.logw = FAKE  # w missing
    assert lib.hs_round(ctypes.byref(a), None) == 1
    a.w = FAKE
    a.R = FAKE  # p, c missing
    assert lib.hs_round(ctypes.byref(a), None) == 1
    assert lib.hs_round(None, None) == 1


def _delayed(lib, **kw):
    a = dict(alpha=FAKE, agree=None, mode=0, B=4, N=8, K=8, count=FAKE, hybrid=0, hist=FAKE,
             clock=FAKE, logw=FAKE, w=FAKE, eta=0.5, R=FAKE, p=FAKE, c=FAKE, loss=None, nloss=None)
    a.update(kw)
    return lib.hs_delayed_update(a["alpha"], a["agree"], a["mode"], a["B"], a["N"], a["K"],
                                 a["count"], a["hybrid"], a["hist"], a["clock"], a["logw"], a["w"],
                                 a["eta"], a["R"], a["p"], a["c"], a["loss"], a["nloss"], None)


def test_delayed_update_validation_codes():
    lib = hs.load_library()
    assert _delayed(lib, B=0) == 2
    assert _delayed(lib, K=0) == 2
    assert _delayed(lib, N=65) == 8
    assert _delayed(lib, K=65) == 8
    assert _delayed(lib, mode=2) == 10
    assert _delayed(lib, alpha=None) == 1
    assert _delayed(lib, mode=1, agree=None) == 1
    assert _delayed(lib, count=None) == 1
    assert _delayed(lib, hist=None) == 1
    assert _delayed(lib, clock=None) == 1
    assert _delayed(lib, w=None) == 1
    assert _delayed(lib, c=None) == 1
    assert _delayed(lib, eta=float("inf")) == 10
    assert _delayed(lib, hybrid=-1) == 10


def _topl(lib, **kw):
    a = dict(target=hs.hs_view(FAKE, 8 * 151936, 151936), N=8, B=1, K=8, V=151936, dtype=1,
             L=10, T=1.0, mode=0, gamma=FAKE, hit=None, children=None, ws=FAKE * 16,
             ws_bytes=1 << 30)
    a.update(kw)
    d = kw.get("drafters", _views(a["N"]))
    tv = a["target"]
    return lib.hs_eval_topl(ctypes.byref(tv) if tv is not None else None, d, a["N"], a["B"],
                            a["K"], a["V"], a["dtype"], a["L"], a["T"], a["mode"], a["gamma"],
                            a["hit"], a["children"], a["ws"], a["ws_bytes"], None)


def test_eval_topl_validation_codes():
    lib = hs.load_library()
    assert lib.hs_eval_topl_workspace_size(1, 8, 8, 151936, 10, 1) > 0
    assert lib.hs_eval_topl_workspace_size(1, 8, 8, 151936, 33, 1) == 0
    assert lib.hs_eval_topl_workspace_size(1, 8, 8, 5, 6, 1) == 0
    assert lib.hs_eval_topl_workspace_size(1, 8, 8, 151936, 10, 7) == 0
    assert _topl(lib, N=0) == 2
    assert _topl(lib, L=0) == 2
    assert _topl(lib, L=33) == 2
    assert _topl(lib, V=9, L=10) == 2
    assert _topl(lib, N=65, drafters=_views(65)) == 8
    assert _topl(lib, dtype=5) == 3
    assert _topl(lib, mode=3) == 10
    assert _topl(lib, target=None) == 1
    assert _topl(lib, drafters=None) == 1
    assert _topl(lib, gamma=None) == 1  # sample mode needs gamma
    assert _topl(lib, mode=1, gamma=None, hit=None) == 1
    assert _topl(lib, T=0.0) == 5
    assert _topl(lib, T=float("inf")) == 5
    assert _topl(lib, target=hs.hs_view(FAKE + 2, 8 * 151936, 151936)) == 4
    assert _topl(lib, drafters=_views(8, sk=3)) == 4
    assert _topl(lib, V=1 << 22) == 8
    assert _topl(lib, ws=None) == 7
    assert _topl(lib, ws_bytes=1000) == 7
    assert _topl(lib, ws=FAKE * 16 + 8) == 4


def test_play_and_regret_validation_codes():
    lib = hs.load_library()
    assert lib.hs_play(FAKE, 0, 8, 0, None, FAKE, None) == 2
    assert lib.hs_play(FAKE, 4, 65, 0, None, FAKE, None) == 8
    assert lib.hs_play(FAKE, 4, 8, 2, None, FAKE, None) == 10
    assert lib.hs_play(None, 4, 8, 0, None, FAKE, None) == 1
    assert lib.hs_play(FAKE, 4, 8, 1, None, FAKE, None) == 1  # sampling needs u
    reg = lambda **kw: lib.hs_regret_update(*[kw.get(k, d) for k, d in (
        ("loss", FAKE), ("L", 1), ("B", 4), ("N", 8), ("played", FAKE), ("cum", FAKE),
        ("pl", FAKE), ("regret", FAKE), ("eal", None), ("eal_sum", None), ("s", None))])
    assert reg(L=0) == 2
    assert reg(B=0) == 2
    assert reg(N=65) == 8
    assert reg(played=None) == 1
    assert reg(regret=None) == 1
    assert reg(eal=FAKE) == 1


def test_binding_constants_match_the_header():
    import os
    import re
    head = open(os.path.join(os.path.dirname(__file__), "..", "include", "hedgespec.h")).read()
    defs = {m.group(1): int(m.group(2)) for m in re.finditer(r"^#define (HS_\w+) (\d+)", head, re.M)}
    pairs = {"HS_OK": hs.HS_OK, "HS_F32": hs.HS_F32, "HS_BF16": hs.HS_BF16,
             "HS_SAMPLE": hs.SAMPLE, "HS_GREEDY": hs.GREEDY, "HS_LOSS_LENGTH": hs.LOSS_LENGTH,
             "HS_LOSS_ACCEPT_TOKEN": hs.LOSS_ACCEPT_TOKEN,
             "HS_LOSS_ACCEPT_CHUNK": hs.LOSS_ACCEPT_CHUNK, "HS_MAX_DRAFTERS": hs.MAX_DRAFTERS,
             "HS_MAX_POSITIONS": hs.MAX_POSITIONS, "HS_MAX_TOPL": hs.MAX_TOPL,
             "HS_PLAY_ARGMAX": hs.PLAY_ARGMAX, "HS_PLAY_SAMPLE": hs.PLAY_SAMPLE}
    for name, value in pairs.items():
        assert defs[name] == value, name


def test_workspace_control_block_layout(tmp_path):
    # the header's statement of the control block (epoch at 0, tagged counters at 16 and 24,
    # mailboxes from 64, aligned disjoint regions) against the library's own layout code,
    # compiled for the host and run on the CPU
    import subprocess

    exe = tmp_path / "ws_layout_check"
    src = os.path.join(ROOT, "tests", "ws_layout_check.cpp")
    subprocess.check_call(["/opt/rocm/bin/hipcc", "-std=c++17", "-O1", "-I",
                           os.path.join(ROOT, "include"), "-I",
                           os.path.join(ROOT, "paper_2510_20064_amd", "csrc"), src, "-o", str(exe)])
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "layout check: ok" in out.stdout


def test_noalloc_workspace_limit_and_validation():
    # hs_eval_alpha_noalloc: its fixed workspace size, a shape that needs more is refused with
    # HS_ERR_WORKSPACE, and an invalid shape gets hs_eval_alpha's own error, all on the host
    # before any HIP call (the pointers are fakes, never dereferenced)
    lib = hs.load_library()
    cap = int(lib.hs_eval_alpha_noalloc_max_workspace())
    assert cap == 64 << 20
    assert lib.hs_eval_alpha_workspace_size(32, 64, 8, 151936, 1) <= cap  # the large pool fits
    assert lib.hs_eval_alpha_workspace_size(64, 64, 8, 151936, 1) > cap

    def call(B, N, K, V, T=1.0):
        tv = hs.hs_view(FAKE, K * 151936, 151936)
        return lib.hs_eval_alpha_noalloc(ctypes.byref(tv), _views(N, sb=K * 151936), N, B, K, V, 1,
                                         T, 0, FAKE, None, None, None, None)

    assert call(64, 64, 8, 151936) == 7  # HS_ERR_WORKSPACE
    assert b"hs_eval_alpha_noalloc" in lib.hs_last_error()
    assert call(0, 8, 8, 151936) == 2  # HS_ERR_SHAPE
    assert call(1, 65, 8, 151936) == 8  # HS_ERR_LIMIT
    assert call(1, 8, 8, 151936, T=0.0) == 5  # HS_ERR_TEMPERATURE


def _cmass(lib, **kw):
    a = dict(target=hs.hs_view(FAKE, 8 * 151936, 151936), N=8, B=1, K=8, V=151936, dtype=1,
             T=0.7, lse=FAKE, cand=FAKE, C=10, gamma=FAKE)
    a.update(kw)
    tv = a["target"]
    return lib.hs_candidate_mass(ctypes.byref(tv) if tv is not None else None, a["N"], a["B"],
                                 a["K"], a["V"], a["dtype"], a["T"], a["lse"], a["cand"], a["C"],
                                 a["gamma"], None)


def test_candidate_mass_validation_codes():
    # every rejection happens on the host, before any HIP call (no GPU here)
    lib = hs.load_library()
    assert _cmass(lib, N=0) == 2
    assert _cmass(lib, K=65) == 8
    assert _cmass(lib, dtype=5) == 3
    assert _cmass(lib, target=None) == 1
    assert _cmass(lib, lse=None) == 1
    assert _cmass(lib, cand=None) == 1
    assert _cmass(lib, gamma=None) == 1
    assert _cmass(lib, C=0) == 8
    assert _cmass(lib, C=1025) == 8
    assert _cmass(lib, T=0.0) == 5
    assert _cmass(lib, T=float("nan")) == 5
    assert _cmass(lib, target=hs.hs_view(FAKE + 2, 8 * 151936, 151936)) == 4
