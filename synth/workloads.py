"""Seeded synthetic inputs for the beam-search output layer.

This module only draws and lays out numbers; it contains none of the
method's arithmetic (no projection, softmax, selection or compaction).
Both the fp64 oracle side and the GPU side consume exactly the arrays
produced here.

Workload shapes follow the paper's output-layer setting (Section 2.2:
target vocabularies of 30k-90k subword units; Section 3: state sizes
256-1024, beams 1-12; Section 4.1: large sentence batches).  The paper's
own speed set (a 50,000-sentence subset of the shared-task training data)
is not available; these seeded draws stand in for it.

Conventions
-----------
* ``h``  : N x H hypothesis states, row-major.
* ``W``  : H x V output weights, row-major (V contiguous).
* ``b``  : V bias, float32.
* ``prev``: N cumulative log-probabilities of the live hypotheses, float32.
* ``off``: S+1 int32 row offsets; rows of sentence s are ``off[s]:off[s+1]``.
* bf16 arrays are carried as ``uint16`` bit patterns (round-to-nearest-even
  from float32), so both sides see identical values.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

SEED_BASE = 180509863


# --------------------------------------------------------------------------
# number formats (data layout only)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return uint16 bits.

    Inputs are finite.  This is the storage format of the half-precision
    workloads; it is not part of the method.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32)


# --------------------------------------------------------------------------
# one decode step
# --------------------------------------------------------------------------
@dataclasses.dataclass
class StepInputs:
    dtype: str            # "f32" or "bf16" (storage type of h and W)
    h: np.ndarray         # N x H float32, or uint16 bf16 bits
    W: np.ndarray         # H x V float32, or uint16 bf16 bits
    b: np.ndarray         # V float32
    prev: np.ndarray      # N float32
    off: np.ndarray       # S+1 int32
    k: int
    name: str = ""
    seed: int = 0

    @property
    def N(self) -> int:
        return int(self.h.shape[0])

    @property
    def H(self) -> int:
        return int(self.h.shape[1])

    @property
    def V(self) -> int:
        return int(self.W.shape[1])

    @property
    def S(self) -> int:
        return int(self.off.shape[0] - 1)


def _normal(g: np.random.Generator, shape, std: float, chunk_rows: int = 64) -> np.ndarray:
    """N(0, std) drawn in float64, returned as float32, generated in row chunks."""
    out = np.empty(shape, dtype=np.float32)
    rows = shape[0]
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        out[r0:r1] = (g.standard_normal((r1 - r0,) + tuple(shape[1:])) * std).astype(np.float32)
    return out


def uniform_offsets(S: int, beam: int) -> np.ndarray:
    return (np.arange(S + 1, dtype=np.int64) * beam).astype(np.int32)


def make_step(N: Optional[int] = None, H: int = 64, V: int = 1000, k: int = 5, *,
              S: Optional[int] = None, beam: Optional[int] = None,
              rows_per_sentence: Optional[list] = None,
              dtype: str = "f32", seed: int = 0, w_std: Optional[float] = None,
              bias: str = "uniform", name: str = "") -> StepInputs:
    """Draw one decode step.

    Draw order is fixed: h, W, b, prev.  ``h ~ N(0,1)``, ``W ~ N(0, w_std)``
    with ``w_std = 1/sqrt(H)`` (standard deviation, giving unit-variance
    logits), ``b ~ U(-0.1, 0.1)`` (or the Zipf-style ``-0.5*ln(j+1)`` when
    ``bias="zipf"``), ``prev ~ U(-5, 0)``.
    """
    if rows_per_sentence is not None:
        rps = [int(r) for r in rows_per_sentence]
        off = np.concatenate([[0], np.cumsum(rps)]).astype(np.int32)
    else:
        if S is None or beam is None:
            raise ValueError("give S and beam, or rows_per_sentence")
        off = uniform_offsets(S, beam)
    n_rows = int(off[-1])
    if N is not None and N != n_rows:
        raise ValueError(f"N={N} does not match offsets total {n_rows}")
    g = np.random.Generator(np.random.PCG64(seed))
    if w_std is None:
        w_std = 1.0 / np.sqrt(H)
    h = _normal(g, (n_rows, H), 1.0)
    W = _normal(g, (H, V), w_std)
    if bias == "uniform":
        b = g.uniform(-0.1, 0.1, size=V).astype(np.float32)
    elif bias == "zipf":
        b = (-0.5 * np.log(np.arange(1, V + 1, dtype=np.float64))).astype(np.float32)
    elif bias == "zero":
        b = np.zeros(V, dtype=np.float32)
    else:
        raise ValueError(bias)
    prev = g.uniform(-5.0, 0.0, size=n_rows).astype(np.float32)
    if dtype == "bf16":
        h = f32_to_bf16_bits(h)
        W = f32_to_bf16_bits(W)
    elif dtype != "f32":
        raise ValueError(dtype)
    return StepInputs(dtype, h, W, b, prev, off, int(k), name=name, seed=seed)


def add_near_ties(inp: StepInputs, frac: float = 0.01, delta: float = 1e-6,
                  seed: int = 0, exact: bool = False) -> StepInputs:
    """Copy a fraction of W columns onto other columns with a tiny bias offset.

    For ``floor(frac*V)`` target columns j2 (drawn without replacement) and
    an unused source column j1 each: ``W[:, j2] = W[:, j1]`` and
    ``b[j2] = b[j1] + s*delta`` with a fair-coin sign s (``delta=0`` when
    ``exact``), so every row gets near-tied (or exactly tied) logit pairs.
    """
    g = np.random.Generator(np.random.PCG64(seed))
    V = inp.V
    n = int(np.floor(frac * V))
    if n == 0:
        return inp
    perm = g.permutation(V)
    j2 = perm[:n]
    j1 = perm[n:2 * n]
    W = inp.W.copy()
    b = inp.b.astype(np.float64).copy()
    W[:, j2] = W[:, j1]
    sign = np.where(g.random(n) < 0.5, -1.0, 1.0)
    b[j2] = b[j1] + (0.0 if exact else 1.0) * sign * delta
    return dataclasses.replace(inp, W=W, b=b.astype(np.float32))


# --------------------------------------------------------------------------
# the five workloads (sizes in the names)
# --------------------------------------------------------------------------
WORKLOADS = [
    dict(name="S1_beam5_H256_V8000_k5_f32", S=1, beam=5, H=256, V=8000, k=5, dtype="f32"),
    dict(name="S64_beam5_H512_V30000_k5_f32_neartie", S=64, beam=5, H=512, V=30000, k=5, dtype="f32",
         near_ties=True),
    dict(name="S128_beam5_H1024_V60000_k5_bf16", S=128, beam=5, H=1024, V=60000, k=5, dtype="bf16"),
    dict(name="S256_beam12_H1024_V90000_k12_bf16_zipf", S=256, beam=12, H=1024, V=90000, k=12,
         dtype="bf16", bias="zipf"),
    dict(name="loop_S512_beam5_H1024_V50000_k5_bf16", S=512, beam=5, H=1024, V=50000, k=5,
         dtype="bf16", T=60, Lmin=5, Lmax=60),
]
SMALL = WORKLOADS[0]["name"]
NEARTIE = WORKLOADS[1]["name"]
V60K = WORKLOADS[2]["name"]
V90K = WORKLOADS[3]["name"]
LOOP = WORKLOADS[4]["name"]


def workload_index(name: str) -> int:
    for i, c in enumerate(WORKLOADS):
        if c["name"] == name:
            return i
    raise KeyError(f"no workload named {name!r}")


def workload_seed(name: str) -> int:
    return SEED_BASE + workload_index(name)


def make_workload(name: str, seed: Optional[int] = None) -> StepInputs:
    """Single-step inputs of a named workload (for the decode-loop workload, its first step)."""
    c = WORKLOADS[workload_index(name)]
    sd = workload_seed(name) if seed is None else seed
    inp = make_step(H=c["H"], V=c["V"], k=c["k"], S=c["S"], beam=c["beam"], dtype=c["dtype"],
                    seed=sd, bias=c.get("bias", "uniform"), name=c["name"])
    if c.get("near_ties"):
        inp = add_near_ties(inp, frac=0.01, delta=1e-6, seed=sd + 1000)
    return inp


# --------------------------------------------------------------------------
# the decode-loop workload: multi-step decode schedule
# --------------------------------------------------------------------------
@dataclasses.dataclass
class LoopWorkload:
    S: int
    beam: int
    H: int
    V: int
    k: int
    T: int
    lengths: np.ndarray   # S int32, target length L_s in [Lmin, Lmax]
    W: np.ndarray         # H x V bf16 bits
    b: np.ndarray         # V float32
    prev0: np.ndarray     # S*beam float32 scores of the step-0 hypotheses
    seed: int

    def h_rows(self, s: int, t: int) -> np.ndarray:
        """bf16 bits of the ``beam`` decoder states of sentence s at step t.

        Regenerated from the seed for each (sentence, step): a stand-in for
        the decoder RNN, whose weights are not available.
        """
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, 7, s, t])))
        x = g.standard_normal((self.beam, self.H)).astype(np.float32)
        return f32_to_bf16_bits(x)

    def h_table(self) -> np.ndarray:
        """All states as a [S, T, beam, H] uint16 array (bf16 bits)."""
        out = np.empty((self.S, self.T, self.beam, self.H), dtype=np.uint16)
        for s in range(self.S):
            for t in range(self.T):
                out[s, t] = self.h_rows(s, t)
        return out

    def alive_after(self, t: int, sentence_ids: np.ndarray) -> np.ndarray:
        """Sentence s is still live after step t iff t < L_s - 1 (EOS forced at L_s - 1)."""
        return (t < self.lengths[np.asarray(sentence_ids)] - 1)


def make_loop_workload(seed: Optional[int] = None, S: Optional[int] = None, V: Optional[int] = None,
                       H: Optional[int] = None, T: Optional[int] = None,
                       Lmin: Optional[int] = None, Lmax: Optional[int] = None) -> LoopWorkload:
    """The decode-loop workload (optionally shrunk for tests): lengths, weights, bias, step-0 scores."""
    c = WORKLOADS[workload_index(LOOP)]
    sd = workload_seed(LOOP) if seed is None else seed
    S = c["S"] if S is None else S
    V = c["V"] if V is None else V
    H = c["H"] if H is None else H
    T = c["T"] if T is None else T
    Lmin = c["Lmin"] if Lmin is None else Lmin
    Lmax = c["Lmax"] if Lmax is None else Lmax
    if not (1 <= Lmin <= Lmax <= T):
        raise ValueError("need 1 <= Lmin <= Lmax <= T")
    g = np.random.Generator(np.random.PCG64(sd))
    lengths = g.integers(Lmin, Lmax + 1, size=S).astype(np.int32)
    W = f32_to_bf16_bits(_normal(g, (H, V), 1.0 / np.sqrt(H)))
    b = g.uniform(-0.1, 0.1, size=V).astype(np.float32)
    prev0 = g.uniform(-5.0, 0.0, size=S * c["beam"]).astype(np.float32)
    return LoopWorkload(S=S, beam=c["beam"], H=H, V=V, k=c["k"], T=T, lengths=lengths,
                        W=W, b=b, prev0=prev0, seed=sd)


# --------------------------------------------------------------------------
# natural end of sentence: a decoder stand-in whose EOS score rises with the step
# --------------------------------------------------------------------------
@dataclasses.dataclass
class EosWorkload:
    S: int
    k: int
    H: int
    V: int
    T: int
    eos: int
    lengths: np.ndarray   # S int32: the step around which each sentence's EOS score overtakes
    W: np.ndarray         # H x V bf16 bits
    b: np.ndarray         # V float32
    gamma: float
    seed: int

    def h_rows(self, s: int, t: int) -> np.ndarray:
        """bf16 bits of the k states of sentence s at step t: N(0, 1) noise plus
        gamma * (t - L_s) along the direction that raises the EOS score by
        exactly that much (W[:, eos] / |W[:, eos]|^2), so hypotheses end around
        their sentence's length, each at its own step."""
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, 11, s, t])))
        x = g.standard_normal((self.k, self.H))
        w = bf16_bits_to_f32(self.W[:, self.eos]).astype(np.float64)
        x = x + self.gamma * (t - float(self.lengths[s])) * (w / np.dot(w, w))[None, :]
        return f32_to_bf16_bits(x.astype(np.float32))

    def h_table(self) -> np.ndarray:
        """All states as a [S, T, k, H] uint16 array (bf16 bits)."""
        out = np.empty((self.S, self.T, self.k, self.H), dtype=np.uint16)
        for s in range(self.S):
            for t in range(self.T):
                out[s, t] = self.h_rows(s, t)
        return out


def make_eos_workload(S: int = 24, k: int = 4, H: int = 128, V: int = 500, T: int = 14, Lmin: int = 2,
                      Lmax: int = 9, eos: int = 3, gamma: float = 3.0, seed: Optional[int] = None) -> EosWorkload:
    """Weights, bias and drawn lengths for a beam search with natural EOS."""
    sd = SEED_BASE + 50 if seed is None else seed
    g = np.random.Generator(np.random.PCG64(sd))
    W = f32_to_bf16_bits(_normal(g, (H, V), 1.0 / np.sqrt(H)))
    b = g.uniform(-0.1, 0.1, V).astype(np.float32)
    lengths = g.integers(Lmin, Lmax + 1, S).astype(np.int32)
    return EosWorkload(S, k, H, V, T, eos, lengths, W, b, gamma, sd)
