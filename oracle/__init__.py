"""Float64 CPU oracle for the HedgeSpec drafter-evaluation path.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the bench's CPU-baseline
leg may import this package; the product library never does. It shares no code
with the GPU path; both sides read the same bytes from the seeded generator.

The arithmetic lives in ``hs_oracle.c`` (plain fp64 loops, one function per
definition in the paper); this module only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hs_oracle.c")
# HS_ORACLE_LIB: a build of hs_oracle.c to load instead (the sanitizer test's instrumented one)
_LIB = os.environ.get("HS_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

F32, BF16, F16 = 0, 1, 2
LOSS_LENGTH, LOSS_ACCEPT_TOKEN, LOSS_ACCEPT_CHUNK = 0, 1, 2
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no fast-math, no fused multiply-add, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
                               "-ffp-contract=off", "-std=c11", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.environ.get("HS_ORACLE_LIB"):
            build()
        lib = ctypes.CDLL(_LIB)
        P, I, I64, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
        lib.or_row_stats.argtypes = [P, I, I64, D, P, P, P]
        lib.or_row_stats.restype = None
        lib.or_alpha.argtypes = [P, P, I, I64, D, D, D]
        lib.or_alpha.restype = D
        lib.or_eval.argtypes = [P, I, I64, I, I64, I64, D, I, P, P, P, P, P]
        lib.or_eval.restype = I
        lib.or_topl.argtypes = [P, I, I64, I, I64, I64, I, D, I, P, P, P]
        lib.or_topl.restype = I
        lib.or_candidate_mass.argtypes = [P, I, I64, I64, I64, I, I, P, D, P]
        lib.or_candidate_mass.restype = I
        lib.or_hybrid_losses.argtypes = [P, I, I, I, I64, P]
        lib.or_hybrid_losses.restype = I
        lib.or_play.argtypes = [P, I, I, I, P, P]
        lib.or_play.restype = None
        lib.or_regret_update.argtypes = [P, I, I, I, P, P, P, P, P, P]
        lib.or_regret_update.restype = None
        lib.or_softmax_stats.argtypes = [P, I, I64, I64, I64, D, P, P, P]
        lib.or_softmax_stats.restype = I
        lib.or_path.argtypes = [P, I, I, P]
        lib.or_path.restype = I
        lib.or_eal_path.argtypes = [P, I]
        lib.or_eal_path.restype = D
        lib.or_accept_len.argtypes = [P, I, I, I, P, P, P, P, I, P]
        lib.or_accept_len.restype = I
        lib.or_hedge.argtypes = [P, P, I, I, I, D]
        lib.or_hedge.restype = None
        lib.or_normalhedge.argtypes = [P, P, P, P, I, I, I]
        lib.or_normalhedge.restype = None
        lib.or_normalhedge_residual.argtypes = [P, I, D]
        lib.or_normalhedge_residual.restype = D
        _lib = lib
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_of(x: np.ndarray) -> int:
    if x.dtype == np.float32:
        return F32
    if x.dtype == np.uint16:
        return BF16
    if x.dtype == np.float16:
        return F16
    raise TypeError("logits must be float32, float16 or uint16 (bf16 bit patterns), got %s"
                    % x.dtype)


def set_threads(n: int) -> None:
    """Limit the OpenMP threads the oracle uses (for single-thread timing)."""
    try:
        gomp = ctypes.CDLL("libgomp.so.1")
        gomp.omp_set_num_threads(ctypes.c_int(int(n)))
    except OSError:
        pass


def row_stats(row: np.ndarray, T: float = 1.0):
    """(max, argmax, lse) of one row of stored logits (float32 or bf16 bits)."""
    row = np.ascontiguousarray(row)
    m, a, l = ctypes.c_double(), ctypes.c_int64(), ctypes.c_double()
    _load().or_row_stats(_p(row), _dtype_of(row), row.shape[-1], T, ctypes.byref(m),
                         ctypes.byref(a), ctypes.byref(l))
    return m.value, a.value, l.value


def alpha_pair(zt: np.ndarray, zi: np.ndarray, T: float = 1.0) -> float:
    """Theorem 1: sum_v min(p_v, q_v) for two rows of stored logits."""
    zt, zi = np.ascontiguousarray(zt), np.ascontiguousarray(zi)
    _, _, lt = row_stats(zt, T)
    _, _, li = row_stats(zi, T)
    return _load().or_alpha(_p(zt), _p(zi), _dtype_of(zt), zt.shape[-1], T, lt, li)


def evaluate(logits: np.ndarray, V: Optional[int] = None, T: float = 1.0, want_alpha: bool = True):
    """Evaluate every drafter on every (query, position) group.

    logits: [R][G][ld] (R = N + 1, row 0 = target) stored logits; any leading group shape
    between R and ld is flattened, e.g. [R][B][K][ld].
    Returns dict with alpha [G..][N], agree [G..][N] (uint8), argmax [G..][R] (int64),
    rmax, rlse [G..][R].
    """
    R = logits.shape[0]
    gshape = logits.shape[1:-1]
    ld = logits.shape[-1]
    V = ld if V is None else V
    G = int(np.prod(gshape)) if gshape else 1
    x = np.ascontiguousarray(logits).reshape(R, G, ld)
    N = R - 1
    alpha = np.full((G, N), np.nan)
    agree = np.zeros((G, N), dtype=np.uint8)
    argmax = np.zeros((G, R), dtype=np.int64)
    rmax = np.zeros((G, R))
    rlse = np.zeros((G, R))
    rc = _load().or_eval(_p(x), _dtype_of(x), ld, R, G, V, T, 1 if want_alpha else 0,
                         _p(alpha), _p(agree), _p(argmax), _p(rmax), _p(rlse))
    if rc != 0:
        raise ValueError("or_eval failed: %d" % rc)
    return {"alpha": alpha.reshape(gshape + (N,)), "agree": agree.reshape(gshape + (N,)),
            "argmax": argmax.reshape(gshape + (R,)), "rmax": rmax.reshape(gshape + (R,)),
            "rlse": rlse.reshape(gshape + (R,))}


def topl(logits: np.ndarray, L: int, V: Optional[int] = None, T: float = 1.0,
         want_mass: bool = True):
    """Theorem 2 (EAGLE): the target's probability mass on each drafter's Top_L tokens.

    logits as in ``evaluate``. Returns dict with gamma [G..][N] (NaN when not want_mass),
    hit [G..][N] (uint8: target argmax in Top_L) and idx [G..][N][L] (Top_L in rank order:
    larger logit first, lower index first among equal logits).
    """
    R = logits.shape[0]
    gshape = logits.shape[1:-1]
    ld = logits.shape[-1]
    V = ld if V is None else V
    G = int(np.prod(gshape)) if gshape else 1
    x = np.ascontiguousarray(logits).reshape(R, G, ld)
    N = R - 1
    gamma = np.full((G, N), np.nan)
    hit = np.zeros((G, N), dtype=np.uint8)
    idx = np.zeros((G, N, L), dtype=np.int32)
    rc = _load().or_topl(_p(x), _dtype_of(x), ld, R, G, V, L, T, 1 if want_mass else 0,
                         _p(gamma), _p(hit), _p(idx))
    if rc != 0:
        raise ValueError("or_topl failed: %d" % rc)
    return {"gamma": gamma.reshape(gshape + (N,)), "hit": hit.reshape(gshape + (N,)),
            "idx": idx.reshape(gshape + (N, L))}


def candidate_mass(target: np.ndarray, cand: np.ndarray, V: Optional[int] = None,
                   T: float = 1.0) -> np.ndarray:
    """Theorem 2 with dynamic pruning: the target's softmax mass on given candidate sets.

    target: [G..][ld] stored logits (one target row per group); cand: [G..][N][C] int32 token
    indices, negative = empty slot. Returns gamma [G..][N] (NaN where an index is >= V).
    """
    gshape = target.shape[:-1]
    ld = target.shape[-1]
    V = ld if V is None else V
    G = int(np.prod(gshape)) if gshape else 1
    x = np.ascontiguousarray(target).reshape(G, ld)
    c = np.ascontiguousarray(np.asarray(cand, dtype=np.int32)).reshape(G, -1, cand.shape[-1])
    N, C = c.shape[1], c.shape[2]
    gamma = np.zeros((G, N))
    rc = _load().or_candidate_mass(_p(x), _dtype_of(x), ld, G, V, N, C, _p(c), T, _p(gamma))
    if rc != 0:
        raise ValueError("or_candidate_mass failed: %d" % rc)
    return gamma.reshape(gshape + (N,))


def softmax_stats(x: np.ndarray, V: Optional[int] = None, T: float = 1.0):
    """Row (max, argmax, lse) for a [rows][ld] tensor of stored logits."""
    x = np.ascontiguousarray(x)
    rows, ld = x.shape
    V = ld if V is None else V
    m = np.zeros(rows)
    a = np.zeros(rows, dtype=np.int64)
    l = np.zeros(rows)
    rc = _load().or_softmax_stats(_p(x), _dtype_of(x), rows, V, ld, T, _p(m), _p(a), _p(l))
    if rc != 0:
        raise ValueError("or_softmax_stats failed: %d" % rc)
    return m, a, l


def eal_path(gamma) -> float:
    """Theorem 3's estimator for the gamma sequence gamma_1..gamma_K along one path."""
    g = np.ascontiguousarray(np.asarray(gamma, dtype=np.float64))
    return _load().or_eal_path(_p(g), len(g))


def path(parent, end: int) -> np.ndarray:
    par = np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    out = np.zeros(len(par) + 1, dtype=np.int32)
    n = _load().or_path(_p(par), len(par), int(end), _p(out))
    if n < 0:
        raise ValueError("bad path")
    return out[:n]


def accept_len(gamma: np.ndarray, parent=None, path_end=None, loss_kind: int = LOSS_LENGTH,
               want_prefix: bool = False):
    """EAL [B][N], optional prefix [B][N][M], and loss [L][B][N] from gamma [B][N][M]."""
    g = np.ascontiguousarray(gamma, dtype=np.float64)
    B, N, M = g.shape
    par = None if parent is None else np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    pe = None if path_end is None else np.ascontiguousarray(np.asarray(path_end, dtype=np.int32))
    eal = np.zeros((B, N))
    prefix = np.zeros((B, N, M)) if want_prefix else None
    L = M if loss_kind == LOSS_ACCEPT_TOKEN else 1
    loss = np.zeros((L, B, N))
    rc = _load().or_accept_len(_p(g), B, N, M, _p(par), _p(pe), _p(eal), _p(prefix), loss_kind,
                               _p(loss))
    return {"eal": eal, "prefix": prefix, "loss": loss, "ok": rc == 0}


def hedge(w: np.ndarray, loss: np.ndarray, eta: float) -> np.ndarray:
    """Hedge update of normalised weights w [B][N] with loss [L][B][N]; returns new w."""
    w = np.array(w, dtype=np.float64, order="C", copy=True)
    loss = np.ascontiguousarray(loss, dtype=np.float64)
    L, B, N = loss.shape
    _load().or_hedge(_p(w), _p(loss), L, B, N, eta)
    return w


def normalhedge(R: np.ndarray, p: np.ndarray, loss: np.ndarray):
    """NormalHedge update; returns (R, p, c) after the L loss vectors."""
    R = np.array(R, dtype=np.float64, order="C", copy=True)
    p = np.array(p, dtype=np.float64, order="C", copy=True)
    loss = np.ascontiguousarray(loss, dtype=np.float64)
    L, B, N = loss.shape
    c = np.zeros(B)
    _load().or_normalhedge(_p(R), _p(p), _p(c), _p(loss), L, B, N)
    return R, p, c


def normalhedge_residual(R_row: np.ndarray, c: float) -> float:
    r = np.ascontiguousarray(R_row, dtype=np.float64)
    return _load().or_normalhedge_residual(_p(r), len(r), c)


def window_losses(gamma: np.ndarray, K: int) -> np.ndarray:
    """Token-level length losses [T - K + 1][N] of a token stream gamma [T][N] (window K)."""
    g = np.ascontiguousarray(gamma, dtype=np.float64)
    T, N = g.shape
    out = np.zeros((max(T - K + 1, 0), N))
    n = _load().or_window_losses(_p(g), T, N, K, _p(out))
    assert n == out.shape[0]
    return out


def play(weights: np.ndarray, how: int = 0, u: Optional[np.ndarray] = None) -> np.ndarray:
    """Drafter choice per query from weights [B][N]: argmax (how 0) or an inverse-CDF sample
    with the uniform draws u [B] (how 1); -1 for a row without positive total weight."""
    w = np.ascontiguousarray(weights, dtype=np.float64)
    B, N = w.shape
    uu = None if u is None else np.ascontiguousarray(u, dtype=np.float64)
    out = np.zeros(B, dtype=np.int32)
    _load().or_play(_p(w), B, N, how, _p(uu), _p(out))
    return out


class Regret:
    """Regret bookkeeping for B queries and N drafters (see or_regret_update)."""

    def __init__(self, B: int, N: int):
        self.cum = np.zeros((B, N))
        self.played = np.zeros(B)
        self.regret = np.zeros(B)
        self.eal_sum = np.zeros(B)

    def update(self, loss: np.ndarray, played: np.ndarray, eal: Optional[np.ndarray] = None):
        """loss [L][B][N] in order, played [L][B] int32 (the drafter played for each vector)."""
        lo = np.ascontiguousarray(loss, dtype=np.float64)
        L, B, N = lo.shape
        pl = np.ascontiguousarray(played, dtype=np.int32).reshape(L, B)
        ea = None if eal is None else np.ascontiguousarray(eal, dtype=np.float64)
        _load().or_regret_update(_p(lo), L, B, N, _p(pl), _p(self.cum), _p(self.played),
                                 _p(self.regret), _p(ea), _p(self.eal_sum if ea is not None else None))
        return self.regret


def hybrid_losses(gamma: np.ndarray, K: int, H: int) -> np.ndarray:
    """Hybrid token losses [n][N] known after the T tokens of gamma [T][N]: acceptance loss for
    the first H tokens, the window-K length loss after them."""
    g = np.ascontiguousarray(gamma, dtype=np.float64)
    T, N = g.shape
    out = np.zeros((T, N))
    n = _load().or_hybrid_losses(_p(g), T, N, K, int(H), _p(out))
    return out[:n]


class QfiD:
    """Queued Full-Information with Delays (Appendix, algorithm QFI-D) with Hedge and
    NormalHedge as base learners, one learner pair per query, fed the token-level length loss
    (or, with hybrid = H > 0, the acceptance loss for each query's first H tokens).

    push(gamma, count): query b's token stream grows by gamma[b, :, :count[b]] (the feedback of
    its next count[b] tokens, [N] each). Every token whose loss is known and not yet used gives
    one loss vector; they enter the FIFO in token order and the base learners take them all, in
    that order, before the next prediction. Returns the loss vectors used per query (a list of
    [L_b][N] arrays)."""

    def __init__(self, B: int, N: int, K: int, eta: float, hybrid: int = 0):
        self.B, self.N, self.K, self.eta, self.hybrid = B, N, K, eta, hybrid
        self.stream = [np.zeros((0, N)) for _ in range(B)]
        self.done = [0] * B  # loss vectors already used
        self.w = np.full((B, N), 1.0 / N)
        self.R = np.zeros((B, N))
        self.p = np.full((B, N), 1.0 / N)
        self.c = np.zeros(B)

    def push(self, gamma: np.ndarray, count):
        used = []
        for b in range(self.B):
            m = int(count[b])
            self.stream[b] = np.concatenate([self.stream[b], np.asarray(gamma[b, :, :m]).T])
            ls = hybrid_losses(self.stream[b], self.K, self.hybrid)[self.done[b]:]
            self.done[b] += ls.shape[0]
            if ls.shape[0]:
                lb = ls[:, None, :]  # [L][1][N]
                self.w[b:b + 1] = hedge(self.w[b:b + 1], lb, self.eta)
                R, p, c = normalhedge(self.R[b:b + 1], self.p[b:b + 1], lb)
                self.R[b:b + 1], self.p[b:b + 1], self.c[b] = R, p, c[0]
            used.append(ls)
        return used
