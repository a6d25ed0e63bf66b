"""Seeded synthetic inputs for the sparse-FFN kernels and for their oracle.

This module holds no FFN arithmetic: it only draws Gaussian tensors, encodes them
as fp32 or bfloat16 bit patterns and names the workload shapes.  Both the GPU
tests/benchmark and the CPU oracle take their inputs from here, so the two sides
see bit-identical data.

Recipe (per weight set, ``seed``):
  numpy ``SeedSequence(seed).spawn(5)`` -> one PCG64 stream per tensor, in the order
  x, (W_gate | A), B, W_up, W_down^T.  Values are float32 standard normals scaled by
  the standard deviation below, then (bf16 weights) rounded to nearest-even bf16.
    x        [T, d]      N(0, 1)
    W_gate   [d_ff, d]   N(0, 1/d)       standard gating
    A        [r, d]      N(0, 1/d)       LoPA V factor
    B        [d_ff, r]   N(0, 1/r)       LoPA U factor
    W_up     [d_ff, d]   N(0, 1/d)
    W_down^T [d_ff, d]   N(0, 1/d_ff)    (row i = output vector of neuron i)
Correlated batches (make_tokens_correlated): x_tau = sqrt(rho) c + sqrt(1 - rho) n_tau with
one common N(0, 1) vector c per batch, so every token is still N(0, 1) (the thresholds
hold) while the active sets of a batch overlap and their union shrinks.
Quantized weight sets (int8 / int4) draw the codes directly: per matrix a PCG64 stream gives
q = clip(rint(N(0, (qmax/3)^2)), -qmax, qmax) with qmax = 127 or 7, then one scale per row,
s_i = std / (qmax/3) * U(0.8, 1.2), so that s_i q_ij has about the standard deviation above.
With these scales every gate pre-activation is close to N(0, 1), so the threshold
t = Phi^-1(s) gives sparsity s: 0, 0.8416, 1.2816, 1.6449 for 50/80/90/95%.
The full FFN form (LoPA's fixed term G, RMSNorm between the factors) takes its extra
inputs from ``make_form``: G's column per row uniform over [0, d), its sign +1 or -1
with equal odds, and RMSNorm gains N(1, 0.25^2).  With G the gate pre-activation is
close to N(0, 2) (B z and x[g_idx[i]] each contribute variance 1; after RMSNorm z has
unit mean square), so the thresholds above scale by sqrt(2).
The paper timed trained checkpoints, which are not available; these Gaussian
weights reproduce the sparsity level but not the correlation of real masks, so
the batched union here is the iid worst case.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

F32 = 0
BF16 = 1
I8 = 2     # int8 codes with an fp32 scale per row
I4 = 3     # int4 codes, two a byte (element 2k in the low nibble), fp32 scale per row
QMAX = {I8: 127, I4: 7}

# activation thresholds for a target sparsity under N(0, 1) gate pre-activations
THRESHOLD = {0.50: 0.0, 0.80: 0.8416, 0.90: 1.2816, 0.95: 1.6449}


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round finite float32 values to the nearest bfloat16 (ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    a = rng.standard_normal(size=shape, dtype=np.float32)
    a *= np.float32(std)
    return a


def _encode(a: np.ndarray, wdt: int) -> np.ndarray:
    return a if wdt == F32 else f32_to_bf16_bits(a)


def pack_int4(q: np.ndarray) -> np.ndarray:
    """int8 codes in [-8, 7], [rows, cols] with cols even -> uint8 [rows, cols/2], element 2k in
    the low nibble of byte k (two's-complement nibbles)."""
    q = np.asarray(q, np.int8)
    lo = q[:, 0::2].astype(np.uint8) & np.uint8(15)
    hi = (q[:, 1::2].astype(np.uint8) & np.uint8(15)) << np.uint8(4)
    return (lo | hi).astype(np.uint8)


def unpack_int4(b: np.ndarray) -> np.ndarray:
    """Inverse of pack_int4."""
    b = np.asarray(b, np.uint8)
    lo = (b & np.uint8(15)).astype(np.int16)
    hi = (b >> np.uint8(4)).astype(np.int16)
    q = np.empty((b.shape[0], 2 * b.shape[1]), np.int16)
    q[:, 0::2], q[:, 1::2] = lo, hi
    return np.where(q >= 8, q - 16, q).astype(np.int8)


def _codes(rng: np.random.Generator, shape, std: float, wdt: int):
    """Quantized matrix of about the given standard deviation: (codes, row scales)."""
    qmax = QMAX[wdt]
    sq = qmax / 3.0
    q = np.clip(np.rint(rng.standard_normal(size=shape, dtype=np.float32) * np.float32(sq)), -qmax, qmax)
    q = q.astype(np.int8)
    s = (np.float32(std / sq) * rng.uniform(0.8, 1.2, size=shape[0]).astype(np.float32)).astype(np.float32)
    return (q if wdt == I8 else pack_int4(q)), s


@dataclass
class FFNInputs:
    x: np.ndarray                  # [T, d] float32
    w_up: np.ndarray               # [d_ff, d] float32 or uint16 (bf16 bits)
    w_down_t: np.ndarray           # [d_ff, d]
    w_gate: np.ndarray | None = None   # [d_ff, d] (standard gating)
    lopa_a: np.ndarray | None = None   # [r, d] (LoPA)
    lopa_b: np.ndarray | None = None   # [d_ff, r] (LoPA)
    wdt: int = BF16
    meta: dict = field(default_factory=dict)
    scales: dict | None = None     # int8 / int4: row scales gate | a, b, up, down (float32)

    @property
    def T(self):
        return self.x.shape[0]

    @property
    def d(self):
        return self.x.shape[1]

    @property
    def d_ff(self):
        return self.w_up.shape[0]

    @property
    def r(self):
        return 0 if self.lopa_a is None else self.lopa_a.shape[0]


def make_inputs(seed: int, T: int, d: int, d_ff: int, *, r: int = 0, wdt: int = BF16) -> FFNInputs:
    """One weight set plus T input tokens; r > 0 selects LoPA factors instead of W_gate."""
    s_x, s_g, s_b, s_u, s_d = (np.random.Generator(np.random.PCG64(s))
                               for s in np.random.SeedSequence(seed).spawn(5))
    x = _normal(s_x, (T, d), 1.0)
    if wdt in QMAX:
        sc = {}
        if r > 0:
            lopa_a, sc["a"] = _codes(s_g, (r, d), d ** -0.5, wdt)
            lopa_b, sc["b"] = _codes(s_b, (d_ff, r), r ** -0.5, wdt)
            w_gate = None
        else:
            w_gate, sc["gate"] = _codes(s_g, (d_ff, d), d ** -0.5, wdt)
            lopa_a = lopa_b = None
        w_up, sc["up"] = _codes(s_u, (d_ff, d), d ** -0.5, wdt)
        w_down_t, sc["down"] = _codes(s_d, (d_ff, d), d_ff ** -0.5, wdt)
        return FFNInputs(x=x, w_up=w_up, w_down_t=w_down_t, w_gate=w_gate, lopa_a=lopa_a, lopa_b=lopa_b,
                         wdt=wdt, meta=dict(seed=seed), scales=sc)
    if r > 0:
        lopa_a = _encode(_normal(s_g, (r, d), d ** -0.5), wdt)
        lopa_b = _encode(_normal(s_b, (d_ff, r), r ** -0.5), wdt)
        w_gate = None
    else:
        w_gate = _encode(_normal(s_g, (d_ff, d), d ** -0.5), wdt)
        lopa_a = lopa_b = None
    w_up = _encode(_normal(s_u, (d_ff, d), d ** -0.5), wdt)
    w_down_t = _encode(_normal(s_d, (d_ff, d), d_ff ** -0.5), wdt)
    return FFNInputs(x=x, w_up=w_up, w_down_t=w_down_t, w_gate=w_gate, lopa_a=lopa_a, lopa_b=lopa_b,
                     wdt=wdt, meta=dict(seed=seed))


@dataclass
class FormInputs:
    g_idx: np.ndarray      # [d_ff] int32, G's column per row, in [0, d)
    g_sign: np.ndarray     # [d_ff] int8, G's value per row, +1 or -1
    rms_gain: np.ndarray   # [r] float32 RMSNorm gains


def make_form(seed: int, d: int, d_ff: int, r: int) -> FormInputs:
    """The extra inputs of the full form, from a stream of their own."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0xF0F1])))
    g_idx = rng.integers(0, d, size=d_ff, dtype=np.int32)
    g_sign = np.where(rng.random(d_ff) < 0.5, -1, 1).astype(np.int8)
    rms_gain = (np.float32(1.0) + _normal(rng, (max(r, 0),), 0.25)).astype(np.float32)
    return FormInputs(g_idx=g_idx, g_sign=g_sign, rms_gain=rms_gain)


def g_repeated_diagonal(d: int, d_ff: int, sign: int = 1):
    """LoPA's fixed term as the repeated diagonal of the appendix on the fixed-matrix
    ablation: row i holds `sign` in column floor(i / k) with k = d_ff / d, read as
    floor(i d / d_ff) when k is not an integer.  Returns (g_idx int32 [d_ff], g_sign int8)."""
    i = np.arange(d_ff, dtype=np.int64)
    return (i * d // d_ff).astype(np.int32), np.full(d_ff, sign, np.int8)


def g_tiled_identity(d: int, d_ff: int):
    """LoPA's fixed term as identity matrices I_d stacked over the d_ff rows (the tiled
    identity of the same ablation): row i holds +1 in column i mod d."""
    return (np.arange(d_ff, dtype=np.int64) % d).astype(np.int32), np.ones(d_ff, np.int8)


def make_tokens_correlated(seed: int, T: int, d: int, rho: float) -> np.ndarray:
    """T tokens sharing a common part: x_tau = sqrt(rho) c + sqrt(1 - rho) n_tau, c and the
    n_tau iid N(0, 1) (each token stays N(0, 1); two tokens correlate by rho)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0xC0C0])))
    c = _normal(rng, (1, d), 1.0)
    n = _normal(rng, (T, d), 1.0)
    return (np.float32(np.sqrt(rho)) * c + np.float32(np.sqrt(1.0 - rho)) * n).astype(np.float32)


def make_tokens(seed: int, T: int, d: int) -> np.ndarray:
    """A separate pool of iid N(0, 1) tokens [T, d] (its own stream, independent of weights)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x70C3])))
    return _normal(rng, (T, d), 1.0)


@dataclass(frozen=True)
class Workload:
    name: str
    d: int
    d_ff: int
    r: int            # 0 = standard gating
    T: int
    wdt: int
    t: float
    seed: int
    n_sets: int
    form: str = ""    # "" the default form; "full": R-S+, SiLU on W_up, G and RMSNorm (LoPA)
    rho: float = 0.0  # token correlation of a batch (0: iid tokens)


# The five workload families; every (sparsity, T) point is its own entry.
def workloads() -> list[Workload]:
    out = [Workload("tiny_f32_std_s90", 256, 1024, 0, 1, F32, THRESHOLD[0.90], 0, 1)]
    for s in (0.50, 0.80, 0.90, 0.95):
        out.append(Workload(f"8b_std_s{int(s * 100)}", 4096, 14336, 0, 1, BF16, THRESHOLD[s], 1000, 4))
    for s in (0.90, 0.95):
        out.append(Workload(f"8b_lopa512_s{int(s * 100)}", 4096, 14336, 512, 1, BF16, THRESHOLD[s], 2000, 4))
    for T in (1, 4, 16, 64):
        out.append(Workload(f"8b_lopa512_s90_T{T}", 4096, 14336, 512, T, BF16, THRESHOLD[0.90], 3000, 4))
    for rho in (0.5, 0.9):
        for T in (16, 64):
            out.append(Workload(f"8b_lopa512_s90_T{T}_rho{int(rho * 10)}", 4096, 14336, 512, T, BF16,
                                THRESHOLD[0.90], 3000, 4, rho=rho))
    for wdt, tag in ((I8, "i8"), (I4, "i4")):
        out.append(Workload(f"8b_std_s90_{tag}", 4096, 14336, 0, 1, wdt, THRESHOLD[0.90], 6000, 4))
        out.append(Workload(f"8b_lopa512_s90_{tag}", 4096, 14336, 512, 1, wdt, THRESHOLD[0.90], 7000, 4))
        out.append(Workload(f"8b_std_s90_{tag}_T4", 4096, 14336, 0, 4, wdt, THRESHOLD[0.90], 6000, 4))
        out.append(Workload(f"8b_lopa512_s90_{tag}_T4", 4096, 14336, 512, 4, wdt, THRESHOLD[0.90], 7000, 4))
    for T in (1, 16):
        out.append(Workload(f"8b_lopa512_full_s90_T{T}", 4096, 14336, 512, T, BF16,
                            round(THRESHOLD[0.90] * 2 ** 0.5, 4), 3000, 4, "full"))
    for T in (1, 8):
        out.append(Workload(f"70b_std_s90_T{T}", 8192, 28672, 0, T, BF16, THRESHOLD[0.90], 4000, 2))
        out.append(Workload(f"70b_lopa1024_s90_T{T}", 8192, 28672, 1024, T, BF16, THRESHOLD[0.90], 5000, 2))
    return out


def workload(name: str) -> Workload:
    for w in workloads():
        if w.name == name:
            return w
    raise KeyError(name)
