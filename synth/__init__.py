"""Seeded synthetic inputs for the drafter-evaluation workloads.

Input plumbing shared by the oracle tests, the GPU parity tests and the bench.
It draws numbers and rounds them to the storage type; it holds none of the
method's arithmetic (no softmax, no acceptance probability, no learner).

The five workloads restate the drafter-evaluation shapes: vocabularies of the
Qwen3 (151936) and Llama-3 (128256) heads, pools of 4 to 64 drafters, chunks
of K = 4..8 verified positions (EAGLE's default chunk is up to 9 tokens,
Appendix "EAGLE's default generation configuration"), greedy and sampled
temperatures, and per-query "domain expert" spread (each drafter is best for
some queries, Section 4.2 and Table 1).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libsynth.so")

F32, BF16, F16 = 0, 1, 2
_lib = None


def build(force: bool = False) -> str:
    """Compile the generator (gcc, OpenMP, no fused multiply-add)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                               "-fno-fast-math", "-std=c11", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        lib.synth_fill.restype = ctypes.c_int
        lib.synth_fill.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                   ctypes.c_int, ctypes.c_int, ctypes.c_uint64, ctypes.c_int64,
                                   ctypes.c_double, ctypes.c_int, ctypes.c_double, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                                   ctypes.c_void_p]
        lib.synth_permutation.restype = None
        lib.synth_permutation.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int, ctypes.c_void_p]
        lib.synth_uniform_int.restype = ctypes.c_int64
        lib.synth_uniform_int.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.c_int64]
        lib.synth_normal.restype = ctypes.c_double
        lib.synth_normal.argtypes = [ctypes.c_uint64, ctypes.c_int64]
        lib.synth_row_key.restype = ctypes.c_uint64
        lib.synth_row_key.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_int64]
        lib.synth_round_f16.restype = ctypes.c_uint16
        lib.synth_round_f16.argtypes = [ctypes.c_double]
        lib.synth_boost_indices.restype = ctypes.c_int
        lib.synth_boost_indices.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                            ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                            ctypes.c_void_p]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# --------------------------------------------------------------------------------------------
# Workload descriptions
# --------------------------------------------------------------------------------------------

SAMPLE, GREEDY = 0, 1
LOSS_LENGTH, LOSS_ACCEPT_TOKEN, LOSS_ACCEPT_CHUNK = 0, 1, 2


@dataclass
class Workload:
    name: str
    B: int
    N: int
    K: int  # chain positions, or tree nodes M
    V: int
    dtype: int
    sigma_t: float
    nboost: int
    boost: float
    scales: List[float]  # s_j, indexed by scale rank j
    permute: bool  # per-query permutation, smallest scale on drafter b mod N
    temperature: float
    mode: int
    loss: int
    eta: float
    seed: int
    rounds: int = 1
    regime_switch: Optional[int] = None  # round at which the scale order reverses
    tree: bool = False
    ld: Optional[int] = None  # row stride in elements (default V)
    extra: dict = field(default_factory=dict)

    @property
    def R(self) -> int:
        return self.N + 1

    @property
    def row_ld(self) -> int:
        return self.ld if self.ld is not None else self.V

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == F32 else 2

    @property
    def input_bytes(self) -> int:
        """Algorithmic bytes of one evaluation: every logit read once."""
        return self.R * self.B * self.K * self.V * self.elem_bytes

    @property
    def positions(self) -> int:
        """Drafter-positions evaluated per round: B * N * K."""
        return self.B * self.N * self.K

    def scale_ranks(self, round: int = 0) -> np.ndarray:
        """[B][N] int: the scale rank j assigned to drafter i at query b in this round."""
        ranks = np.empty((self.B, self.N), dtype=np.int32)
        for b in range(self.B):
            if self.permute:
                perm = np.empty(self.N, dtype=np.int32)
                _load().synth_permutation(self.seed, 0x7065726D, b, self.N, _ptr(perm))
                # smallest scale (rank 0) on drafter b mod N
                j0 = int(np.nonzero(perm == 0)[0][0])
                tgt = b % self.N
                perm[j0], perm[tgt] = perm[tgt], perm[j0]
                ranks[b] = perm
            else:
                ranks[b] = np.arange(self.N, dtype=np.int32)
        if self.regime_switch is not None and round >= self.regime_switch:
            ranks = (self.N - 1) - ranks
        return ranks

    def scale_matrix(self, round: int = 0) -> np.ndarray:
        s = np.asarray(self.scales, dtype=np.float64)
        return s[self.scale_ranks(round)]

    def parent(self) -> Optional[np.ndarray]:
        """Parent array of the draft tree (None for a chain)."""
        if not self.tree:
            return None
        return tree_parents(self.extra["branching"], self.K)

    def path_end(self) -> Optional[np.ndarray]:
        if not self.tree:
            return None
        par = self.parent()
        return seeded_descent(par, self.B, self.seed)


def log_spaced(lo: float, ratio: float, n: int) -> List[float]:
    """s_j = lo * ratio**(j/(n-1)), j = 0..n-1."""
    if n == 1:
        return [lo]
    return [lo * ratio ** (j / (n - 1)) for j in range(n)]


def tree_parents(branching: Sequence[int], M: int) -> np.ndarray:
    """BFS parent array: root, then each level's nodes get `branching[l]` children, truncated to M."""
    par = [-1]
    level = [0]
    for br in branching:
        nxt = []
        for p in level:
            for _ in range(br):
                if len(par) < M:
                    nxt.append(len(par))
                    par.append(p)
        level = nxt
        if len(par) >= M:
            break
    if len(par) != M:
        raise ValueError("branching does not reach M nodes")
    return np.asarray(par, dtype=np.int32)


def seeded_descent(parent: np.ndarray, B: int, seed: int) -> np.ndarray:
    """path_end[b]: from the root pick a uniform child at each node until a node without children."""
    M = len(parent)
    children = [[] for _ in range(M)]
    for n in range(1, M):
        children[parent[n]].append(n)
    out = np.empty(B, dtype=np.int32)
    for b in range(B):
        n, depth = 0, 0
        while children[n]:
            j = _load().synth_uniform_int(seed, 0x70617468, b, depth, len(children[n]))
            n = children[n][j]
            depth += 1
        out[b] = n
    return out


def workloads() -> dict:
    """The five drafter-evaluation workloads, keyed by name."""
    ws = {}
    ws["tiny_chain"] = Workload(
        name="tiny_chain", B=1, N=4, K=4, V=32000, dtype=F32, sigma_t=2.0, nboost=0, boost=0.0,
        scales=[0.1, 0.5, 1.0, 2.0], permute=False, temperature=1.0, mode=SAMPLE,
        loss=LOSS_ACCEPT_TOKEN, eta=0.5, seed=0)
    ws["qwen3_8b_single"] = Workload(
        name="qwen3_8b_single", B=1, N=8, K=8, V=151936, dtype=BF16, sigma_t=3.0, nboost=20,
        boost=8.0, scales=log_spaced(0.2, 20.0, 8), permute=False, temperature=1.0, mode=SAMPLE,
        loss=LOSS_LENGTH, eta=0.5, seed=1)
    ws["batched_serving"] = Workload(
        name="batched_serving", B=64, N=8, K=6, V=128256, dtype=BF16, sigma_t=2.0, nboost=0,
        boost=0.0, scales=log_spaced(0.1, 20.0, 8), permute=True, temperature=0.7, mode=SAMPLE,
        loss=LOSS_LENGTH, eta=0.5, seed=2)
    ws["draft_tree"] = Workload(
        name="draft_tree", B=16, N=16, K=64, V=151936, dtype=BF16, sigma_t=3.0, nboost=20,
        boost=8.0, scales=log_spaced(0.2, 20.0, 16), permute=True, temperature=1.0, mode=SAMPLE,
        loss=LOSS_LENGTH, eta=0.5, seed=3, tree=True, extra={"branching": [3, 2, 2, 2, 1]})
    ws["large_pool_stream"] = Workload(
        name="large_pool_stream", B=32, N=64, K=8, V=151936, dtype=BF16, sigma_t=3.0, nboost=20,
        boost=8.0, scales=log_spaced(0.2, 20.0, 64), permute=True, temperature=1.0, mode=SAMPLE,
        loss=LOSS_LENGTH, eta=math.sqrt(8.0 * math.log(64) / 1000.0), seed=4, rounds=1000,
        regime_switch=500)
    return ws


def variant(w: Workload, **kw) -> Workload:
    """A copy of a workload with some fields changed (reduced sizes for full-check tests)."""
    d = dict(w.__dict__)
    d.update(kw)
    return Workload(**d)


# --------------------------------------------------------------------------------------------
# Generation
# --------------------------------------------------------------------------------------------

def generate(w: Workload, round: int = 0, rows: Optional[Sequence[int]] = None,
             bk: Optional[Sequence[Sequence[int]]] = None, out: Optional[np.ndarray] = None
             ) -> np.ndarray:
    """Logits of one round.

    Returns an array of shape [len(rows)][B][K][ld] (bk None) or [len(rows)][len(bk)][ld],
    uint16 (bf16 bit patterns), float16 or float32. Only the first V entries of each row are written
    (padding beyond V is zero). rows defaults to all N+1 rows (0 = target, 1+i = drafter i).
    """
    lib = _load()
    rows_a = np.asarray(list(range(w.R)) if rows is None else list(rows), dtype=np.int32)
    if bk is None:
        shape = (len(rows_a), w.B, w.K, w.row_ld)
        bk_a, nbk = None, w.B * w.K
    else:
        bk_a = np.ascontiguousarray(np.asarray(bk, dtype=np.int32).reshape(-1, 2))
        nbk = bk_a.shape[0]
        shape = (len(rows_a), nbk, w.row_ld)
    dt = {F32: np.float32, BF16: np.uint16, F16: np.float16}[w.dtype]
    if out is None:
        out = np.zeros(shape, dtype=dt)
    else:
        assert out.shape == shape and out.dtype == dt and out.flags.c_contiguous
    scale = np.ascontiguousarray(w.scale_matrix(round), dtype=np.float64)
    rc = lib.synth_fill(w.dtype, w.V, w.row_ld, w.B, w.K, w.N, w.seed, round, w.sigma_t,
                        w.nboost, w.boost, _ptr(scale), _ptr(rows_a), len(rows_a),
                        None if bk_a is None else _ptr(bk_a), nbk, _ptr(out))
    if rc != 0:
        raise ValueError("synth_fill failed: %d" % rc)
    return out


def bf16_bits_to_f64(a: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) exactly to float64."""
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def decode(w: Workload, a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f64(a) if w.dtype == BF16 else a.astype(np.float64)


def round_f16(x: float) -> int:
    """The binary16 bit pattern the generator stores for the fp64 value x (via fp32)."""
    return int(_load().synth_round_f16(float(x)))


def synthetic_losses(seed: int, rounds: int, L: int, B: int, N: int) -> np.ndarray:
    """Seeded losses in [0, 1], shape [rounds][L][B][N] (learner-stream inputs)."""
    rng = np.random.Generator(np.random.Philox(seed))
    base = rng.uniform(0.0, 1.0, size=(B, N))
    noise = rng.uniform(-0.25, 0.25, size=(rounds, L, B, N))
    return np.clip(base[None, None] + noise, 0.0, 1.0)
