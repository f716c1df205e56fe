"""Seeded synthetic SeKV caches (stored inputs of one decode step).

Everything here is input synthesis.  The values come from a counter-based
generator so that any slice of any cache can be regenerated exactly, on any
machine, in any order and from any number of threads:

* key    = chain of splitmix64 finalisers over (seed, variant, layer, stream, b, g)
* z[i]   = splitmix64 finaliser of (key + i * 0x9E3779B97F4A7C15)   (mod 2**64)
* normal = NTAB[z >> 48], NTAB[j] = Phi^-1((j + 0.5) / 65536)  (tails cut at 4.32 sigma)
* uniform= (z >> 11) * 2**-53

The splitmix64 finaliser is the published mixing function of Steele, Lea and
Flood ("Fast splittable pseudorandom number generators", OOPSLA 2014) with
Vigna's constants.

Storage rounding: every stored value is computed in float64 and rounded once
to the storage type (float32, or bfloat16 with round-to-nearest-even, done as
float64 -> float32 with round-to-odd -> bfloat16 with round-to-nearest-even,
which is a correct single rounding since float32 carries more than 8 + 2 bits).

Span partition (one per sequence, shared by every layer and head): the first
``n_prefix_anchors`` tokens and the last ``window`` tokens are kept at full
resolution; the tokens between are cut left to right into spans whose lengths
are drawn i.i.d. (uniform integers, or ``min(hi, floor(exp(u)))`` with
``u ~ U(ln lo, ln(hi + 1))`` for the log-uniform law); a final remainder
shorter than ``span_min`` joins the full-resolution set, as spans shorter than
the minimum length stay at full resolution in the paper (Sec. 3.2, low-rank
basis paragraph).

Span summaries are the means of the span's reconstructed keys and values (the
workload definition), formed in float64 from the already-rounded stored factors
as (1/|S|) (1^T U) diag(sigma) V^T and then rounded to storage.

Factor arena: one block per (b, kv head, span), in (b, g, S) order, each block
starting on a 256-byte boundary and laid out as
``U_K[|S|][r] | sigma_K[r] | Vt_K[r][d] | U_V[|S|][r] | sigma_V[r] | Vt_V[r][d]``
in the storage type.  ``block_off[b][g][S]`` is the block's byte offset.
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

try:  # inverse normal CDF for the quantile table
    from scipy.special import ndtri as _ndtri
except Exception:  # pragma: no cover - scipy is present in this image
    from statistics import NormalDist

    def _ndtri(p):
        nd = NormalDist()
        return np.array([nd.inv_cdf(float(x)) for x in np.ravel(p)])


_MASK64 = (1 << 64) - 1
_GOLDEN_I = 0x9E3779B97F4A7C15
_GOLDEN = np.uint64(_GOLDEN_I)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_S30, _S27, _S31 = np.uint64(30), np.uint64(27), np.uint64(31)
_S48, _S11 = np.uint64(48), np.uint64(11)

NTAB = _ndtri((np.arange(65536, dtype=np.float64) + 0.5) / 65536.0)

_CHUNK = 1 << 20

# stream ids
ST_PART, ST_Q, ST_AK, ST_AV = 1, 2, 3, 4
ST_UK, ST_SK, ST_VK, ST_UV, ST_SV, ST_VV = 5, 6, 7, 8, 9, 10
ST_NEEDLE = 11
ST_PROJ, ST_TAU, ST_RANK = 12, 13, 14

VARIANTS = {"L": 0, "N": 1}
PLANT_DELTA = 6.0


def _mix_int(x: int) -> int:
    x &= _MASK64
    x ^= x >> 30
    x = (x * 0xBF58476D1CE4E5B9) & _MASK64
    x ^= x >> 27
    x = (x * 0x94D049BB133111EB) & _MASK64
    x ^= x >> 31
    return x


def stream_key(*parts: int) -> int:
    k = 0
    for p in parts:
        k = _mix_int(k + _GOLDEN_I * (int(p) + 1))
    return k


def _hash_block(key: int, start: int, n: int) -> np.ndarray:
    z = np.arange(start, start + n, dtype=np.uint64)
    z *= _GOLDEN
    z += np.uint64(key)
    z ^= z >> _S30
    z *= _M1
    z ^= z >> _S27
    z *= _M2
    z ^= z >> _S31
    return z


def normals(key: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        out[s:s + m] = NTAB[(_hash_block(key, s, m) >> _S48).astype(np.intp)]
    return out


def uniforms(key: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        out[s:s + m] = (_hash_block(key, s, m) >> _S11).astype(np.float64) * (2.0 ** -53)
    return out


# ---------------------------------------------------------------------------
# storage types
# ---------------------------------------------------------------------------

def f64_to_bf16_bits(x) -> np.ndarray:
    """Round float64 to bfloat16 (nearest-even), returned as uint16 bit patterns."""
    x = np.asarray(x, dtype=np.float64)
    flat = x.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)
    for s0 in range(0, flat.size, _CHUNK):
        xc = flat[s0:s0 + _CHUNK]
        f = xc.astype(np.float32)
        back = f.astype(np.float64)
        inexact = back != xc
        over = inexact & (np.abs(back) > np.abs(xc))
        fb = f.view(np.uint32) - over.astype(np.uint32)   # truncate toward zero
        fb |= inexact.astype(np.uint32)                   # sticky bit: round-to-odd
        fb += ((fb >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
        out[s0:s0 + _CHUNK] = (fb >> np.uint32(16)).astype(np.uint16)
    return out.reshape(x.shape)


def bf16_bits_to_f64(b) -> np.ndarray:
    b = np.asarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def to_storage(x64: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(x64, dtype=np.float64).astype(np.float32)
    if dtype == "bf16":
        return f64_to_bf16_bits(x64)
    raise ValueError(dtype)


def from_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    raise ValueError(dtype)


def elem_bytes(dtype: str) -> int:
    return {"f32": 4, "bf16": 2}[dtype]


def _np_storage_type(dtype: str):
    return {"f32": np.float32, "bf16": np.uint16}[dtype]


# ---------------------------------------------------------------------------
# specs
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class CaseSpec:
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rank: int
    top_k: int
    context: int
    n_prefix_anchors: int
    window: int
    span_dist: str          # "uniform" | "loguniform"
    span_min: int
    span_max: int
    dtype: str              # "f32" | "bf16"
    factor_kind: str        # "orthonormal" | "gaussian"
    n_layers: int = 1
    seed: int = 0
    host_factors: bool = False   # factors live in pinned host memory (tier case)
    rank_mode: str = "fixed"     # "fixed": every block has `rank`; "adaptive": per-block ranks

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


WORKLOADS = {
    "tiny-f32": CaseSpec("tiny-f32", batch=1, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8,
                top_k=2, context=2048, n_prefix_anchors=32, window=0,
                span_dist="uniform", span_min=16, span_max=64, dtype="f32",
                factor_kind="orthonormal", seed=1),
    "llama3-8b-layer-32k": CaseSpec("llama3-8b-layer-32k", batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128,
                rank=16, top_k=8, context=32768, n_prefix_anchors=256, window=512,
                span_dist="uniform", span_min=32, span_max=256, dtype="bf16",
                factor_kind="gaussian", seed=2),
    "llama3-8b-layer-128k-b4": CaseSpec("llama3-8b-layer-128k-b4", batch=4, n_q_heads=32, n_kv_heads=8, head_dim=128,
                rank=32, top_k=16, context=131072, n_prefix_anchors=256, window=512,
                span_dist="loguniform", span_min=32, span_max=512, dtype="bf16",
                factor_kind="gaussian", seed=3),
    "llama3-8b-32layer-32k-b32": CaseSpec("llama3-8b-32layer-32k-b32", batch=32, n_q_heads=32, n_kv_heads=8,
                head_dim=128, rank=16, top_k=8, context=32768, n_prefix_anchors=256,
                window=512, span_dist="uniform", span_min=32, span_max=256, dtype="bf16",
                factor_kind="gaussian", n_layers=32, seed=4),
    "llama3-8b-layer-128k-b4-hosttier": CaseSpec("llama3-8b-layer-128k-b4-hosttier", batch=4, n_q_heads=32, n_kv_heads=8,
                head_dim=128, rank=32, top_k=16, context=131072, n_prefix_anchors=256,
                window=512, span_dist="loguniform", span_min=32, span_max=512,
                dtype="bf16", factor_kind="gaussian", seed=3, host_factors=True),
}


def custom_spec(**kw) -> CaseSpec:
    """A small spec for tests; defaults follow the tiny fp32 case."""
    base = dict(name="custom", batch=1, n_q_heads=4, n_kv_heads=2, head_dim=64, rank=8,
                top_k=2, context=512, n_prefix_anchors=8, window=0, span_dist="uniform",
                span_min=8, span_max=32, dtype="f32", factor_kind="gaussian", seed=99)
    base.update(kw)
    return CaseSpec(**base)


# ---------------------------------------------------------------------------
# case container
# ---------------------------------------------------------------------------

@dataclass
class Case:
    spec: CaseSpec
    layer: int
    variant: str
    q: np.ndarray              # [B][Hq][d]            storage type
    anchor_k: np.ndarray       # [B][Hkv][A_max][d]
    anchor_v: np.ndarray
    n_anchors: np.ndarray      # [B] int32
    sum_k: np.ndarray          # [B][Hkv][M_max][d]
    sum_v: np.ndarray
    n_spans: np.ndarray        # [B] int32
    span_len: np.ndarray       # [B][M_max] int32 (0 past n_spans)
    span_logsize: np.ndarray   # [B][M_max] float64 ln|S| (0 past n_spans)
    factors: np.ndarray        # uint8 arena
    block_off: np.ndarray      # [B][Hkv][M_max] int64 byte offsets
    needles: np.ndarray = field(default=None)   # [B][Hkv][n_p] planted spans (variant N)
    block_rank: np.ndarray = field(default=None)  # [B][Hkv][M_max] int32 r_K | r_V << 16, or None

    @property
    def dtype(self) -> str:
        return self.spec.dtype

    @property
    def max_anchors(self) -> int:
        return self.anchor_k.shape[2]

    @property
    def max_spans(self) -> int:
        return self.sum_k.shape[2]

    @property
    def max_span_len(self) -> int:
        return int(self.span_len.max()) if self.span_len.size else 1

    def dims(self) -> dict:
        s = self.spec
        return dict(batch=s.batch, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                    head_dim=s.head_dim, rank=s.rank, top_k=s.top_k,
                    max_anchors=self.max_anchors, max_spans=self.max_spans,
                    max_span_len=max(self.max_span_len, 1), dtype=s.dtype,
                    softmax_scale=s.softmax_scale)


# ---------------------------------------------------------------------------
# partition
# ---------------------------------------------------------------------------

def span_lengths(spec: CaseSpec, b: int):
    """Span lengths of sequence b and the short remainder kept at full resolution."""
    middle = spec.context - spec.n_prefix_anchors - spec.window
    if middle < 0:
        raise ValueError("context shorter than anchors + window")
    n_draw = middle // max(spec.span_min, 1) + 2
    u = uniforms(stream_key(spec.seed, ST_PART, b), n_draw)
    lo, hi = spec.span_min, spec.span_max
    if spec.span_dist == "uniform":
        drawn = lo + np.floor(u * (hi - lo + 1)).astype(np.int64)
    elif spec.span_dist == "loguniform":
        a, c = math.log(lo), math.log(hi + 1)
        drawn = np.minimum(hi, np.floor(np.exp(a + u * (c - a))).astype(np.int64))
    else:
        raise ValueError(spec.span_dist)
    lengths = []
    pos = 0
    for L in drawn:
        rem = middle - pos
        if rem < lo:
            break
        L = int(min(L, rem))
        lengths.append(L)
        pos += L
    return lengths, middle - pos


def block_bytes(length: int, rank: int, head_dim: int, dtype: str, rank_v: int | None = None) -> int:
    rv = rank if rank_v is None else rank_v
    raw = ((length + 1 + head_dim) * (rank + rv)) * elem_bytes(dtype)
    return (raw + 255) // 256 * 256


def rank_granule(dtype: str) -> int:
    """Ranks of adaptive-rank blocks are multiples of this: one 16-byte vector of a U row."""
    return 16 // elem_bytes(dtype)


def draw_ranks(spec: CaseSpec, vkey, b: int, g: int, m: int):
    """Retained ranks (r_K, r_V) of the m spans of (b, g).

    The trained rank-gate predictor is not available; as its stand-in each side keeps
    a uniformly drawn number of granules in [1, rank / granule] of its leading
    components (sigma is sorted descending, so the dropped ones are the smallest)."""
    gr = rank_granule(spec.dtype)
    nmax = max(1, spec.rank // gr)
    u = uniforms(stream_key(*vkey, ST_RANK, b, g), 2 * m).reshape(2, m)
    n = np.minimum(nmax, 1 + np.floor(u * nmax).astype(np.int64))
    return (n[0] * gr).astype(np.int64), (n[1] * gr).astype(np.int64)


# ---------------------------------------------------------------------------
# factor synthesis
# ---------------------------------------------------------------------------

def _orthonormal_cols(mat: np.ndarray) -> np.ndarray:
    """Q of a thin QR with a positive diagonal of R (first column keeps its direction)."""
    qm, rm = np.linalg.qr(mat)
    sgn = np.sign(np.diag(rm))
    sgn[sgn == 0] = 1.0
    return qm * sgn


def _pair_factors(spec: CaseSpec, vkey, b, g, lens, planted, qbar):
    """Float64 factors of every span of (b, g) before storage rounding."""
    r, d, m = spec.rank, spec.head_dim, len(lens)
    sum_l = int(sum(lens))
    fs = 1.0 / math.sqrt(d)
    out = {}
    for side, (su, ss, sv) in (("K", (ST_UK, ST_SK, ST_VK)), ("V", (ST_UV, ST_SV, ST_VV))):
        if spec.factor_kind == "gaussian":
            scale = 1.0 if (side == "V" and planted) else fs
            U = normals(stream_key(*vkey, su, b, g), sum_l * r).reshape(sum_l, r) * scale
            s = np.abs(normals(stream_key(*vkey, ss, b, g), m * r).reshape(m, r))
            s = -np.sort(-s, axis=1) * scale
            Vt = normals(stream_key(*vkey, sv, b, g), m * r * d).reshape(m, r, d) * scale
        elif spec.factor_kind == "orthonormal":
            raw_u = normals(stream_key(*vkey, su, b, g), sum_l * r).reshape(sum_l, r)
            raw_v = normals(stream_key(*vkey, sv, b, g), m * d * r).reshape(m, d, r)
            uu = uniforms(stream_key(*vkey, ss, b, g), m * r).reshape(m, r)
            expo = -np.log1p(-uu)                 # Exp(1) by inversion
            s = -np.sort(-expo, axis=1)           # descending
            U = np.empty_like(raw_u)
            Vt = np.empty((m, r, d))
            start = 0
            for j, L in enumerate(lens):
                U[start:start + L] = _orthonormal_cols(raw_u[start:start + L])
                Vt[j] = _orthonormal_cols(raw_v[j]).T
                start += L
        else:
            raise ValueError(spec.factor_kind)
        out[side] = [U, s, Vt]
    return out


def _plant(spec: CaseSpec, fac, lens, needles, qbar):
    """Make each needle span's keys align with the group's mean query (K side only)."""
    r, d = spec.rank, spec.head_dim
    U, s, Vt = fac["K"]
    nq = float(np.linalg.norm(qbar))
    direction = qbar / nq
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    for j in needles:
        L = lens[j]
        rows = slice(starts[j], starts[j] + L)
        if spec.factor_kind == "orthonormal":
            mu = U[rows].copy()
            mu[:, 0] = 1.0 / math.sqrt(L)
            U[rows] = _orthonormal_cols(mu)
            mv = Vt[j].T.copy()
            mv[:, 0] = direction
            Vt[j] = _orthonormal_cols(mv).T
        else:
            U[rows, 0] = 1.0 / math.sqrt(L)
            Vt[j, 0] = direction
        s[j, 0] = PLANT_DELTA * math.sqrt(L) / (spec.softmax_scale * nq)
        s[j] = -np.sort(-s[j])


def _write_pair(spec, arena_e, eoff, lens, fac_st, ranks=None):
    """Copy the stored factors of one (b, g) into the arena (element view): the leading
    r_K / r_V components of each span (all `rank` of them without a rank table)."""
    d = spec.head_dim
    start = 0
    for j, L in enumerate(lens):
        o = int(eoff[j])
        rows = slice(start, start + L)
        for si, side in enumerate(("K", "V")):
            U, sg, Vt = fac_st[side]
            r = spec.rank if ranks is None else int(ranks[si][j])
            arena_e[o:o + L * r] = U[rows, :r].reshape(-1)
            o += L * r
            arena_e[o:o + r] = sg[j, :r]
            o += r
            arena_e[o:o + r * d] = Vt[j, :r].reshape(-1)
            o += r * d
        start += L


def _span_means(U, s, Vt, lens):
    """(1/|S|) (1^T U) diag(sigma) V^T per span, float64."""
    lens_a = np.asarray(lens, dtype=np.int64)
    starts = np.concatenate([[0], np.cumsum(lens_a)[:-1]]).astype(np.int64)
    colsum = np.add.reduceat(U, starts, axis=0)
    coef = colsum / lens_a[:, None] * s
    return np.einsum("mr,mrd->md", coef, Vt)


def make_case(spec: CaseSpec, layer: int = 0, variant: str = "L", threads: int | None = None,
              arena_out: np.ndarray | None = None, needle_layer: int | None = None) -> Case:
    """Build the stored inputs of one layer of a decode step.

    needle_layer (variant N): draw the planted spans' positions as for that layer, so that
    layers built with the same needle_layer plant the same spans (their keys and values
    are still this layer's own): a stand-in for spans that many layers attend to."""
    if variant not in VARIANTS:
        raise ValueError(variant)
    planted = variant == "N"
    B, Hq, Hkv, d, r = spec.batch, spec.n_q_heads, spec.n_kv_heads, spec.head_dim, spec.rank
    if Hq % Hkv:
        raise ValueError("n_q_heads must be a multiple of n_kv_heads")
    G = Hq // Hkv
    dt = spec.dtype
    e = elem_bytes(dt)
    vkey = (spec.seed, VARIANTS[variant], layer)

    parts = [span_lengths(spec, b) for b in range(B)]
    n_spans = np.array([len(p[0]) for p in parts], dtype=np.int32)
    n_anch = np.array([spec.n_prefix_anchors + p[1] + spec.window for p in parts], dtype=np.int32)
    M_max = max(int(n_spans.max()) if B else 0, 1)
    A_max = max(int(n_anch.max()) if B else 0, 1)
    span_len = np.zeros((B, M_max), dtype=np.int32)
    for b, (lens, _) in enumerate(parts):
        span_len[b, :len(lens)] = lens
    span_logsize = np.zeros((B, M_max), dtype=np.float64)
    nz = span_len > 0
    span_logsize[nz] = np.log(span_len[nz].astype(np.float64))

    qscale = 1.0 if spec.factor_kind == "orthonormal" else 1.0 / math.sqrt(d)
    q64 = np.stack([normals(stream_key(*vkey, ST_Q, b), Hq * d).reshape(Hq, d)
                    for b in range(B)]) * qscale if B else np.zeros((0, Hq, d))
    q_st = to_storage(q64, dt)
    q_dec = from_storage(q_st, dt)

    # retained ranks and block offsets
    adaptive = spec.rank_mode == "adaptive"
    if spec.rank_mode not in ("fixed", "adaptive"):
        raise ValueError(spec.rank_mode)
    ranks = {}
    block_rank = np.zeros((B, Hkv, M_max), dtype=np.int32) if adaptive else None
    block_off = np.zeros((B, Hkv, M_max), dtype=np.int64)
    total = 0
    for b, (lens, _) in enumerate(parts):
        for g in range(Hkv):
            if not len(lens):
                continue
            if adaptive:
                rk, rv = draw_ranks(spec, vkey, b, g, len(lens))
                ranks[(b, g)] = (rk, rv)
                block_rank[b, g, :len(lens)] = (rk | (rv << 16)).astype(np.int32)
                sizes = np.array([block_bytes(L, int(a), d, dt, int(c)) for L, a, c in zip(lens, rk, rv)],
                                 dtype=np.int64)
            else:
                sizes = np.array([block_bytes(L, r, d, dt) for L in lens], dtype=np.int64)
            block_off[b, g, :len(lens)] = total + np.concatenate([[0], np.cumsum(sizes)[:-1]])
            total += int(sizes.sum())
    total = max(total, 256)
    if arena_out is not None:
        if arena_out.nbytes < total or arena_out.dtype != np.uint8:
            raise ValueError("arena_out too small or not uint8")
        arena = arena_out[:total]
    else:
        arena = np.zeros(total, dtype=np.uint8)
    arena_e = arena.view(_np_storage_type(dt))

    st_t = _np_storage_type(dt)
    anchor_k = np.zeros((B, Hkv, A_max, d), dtype=st_t)
    anchor_v = np.zeros((B, Hkv, A_max, d), dtype=st_t)
    sum_k = np.zeros((B, Hkv, M_max, d), dtype=st_t)
    sum_v = np.zeros((B, Hkv, M_max, d), dtype=st_t)
    n_p = max(1, spec.top_k // 2)
    needles = np.full((B, Hkv, n_p), -1, dtype=np.int32) if planted else None

    ascale = qscale
    vscale_anchor = 1.0 if (planted and spec.factor_kind == "gaussian") else ascale

    def work(bg):
        b, g = bg
        lens, _ = parts[b]
        A = int(n_anch[b])
        ak = normals(stream_key(*vkey, ST_AK, b, g), A * d).reshape(A, d) * ascale
        av = normals(stream_key(*vkey, ST_AV, b, g), A * d).reshape(A, d) * vscale_anchor
        anchor_k[b, g, :A] = to_storage(ak, dt)
        anchor_v[b, g, :A] = to_storage(av, dt)
        m = len(lens)
        if m == 0:
            return
        qbar = q_dec[b, g * G:(g + 1) * G].mean(axis=0)
        fac = _pair_factors(spec, vkey, b, g, lens, planted, qbar)
        if planted:
            nkey = vkey if needle_layer is None else (spec.seed, VARIANTS[variant], needle_layer)
            h = uniforms(stream_key(*nkey, ST_NEEDLE, b, g), m)
            chosen = np.sort(np.argsort(h, kind="stable")[:min(n_p, m)])
            needles[b, g, :len(chosen)] = chosen
            _plant(spec, fac, lens, chosen, qbar)
        fac_st = {side: [to_storage(x, dt) for x in fac[side]] for side in fac}
        rk_rv = ranks.get((b, g))
        _write_pair(spec, arena_e, block_off[b, g, :m] // e, lens, fac_st, rk_rv)
        for si, (side, dst) in enumerate((("K", sum_k), ("V", sum_v))):
            U, s, Vt = (from_storage(x, dt) for x in fac_st[side])
            if rk_rv is not None:
                s = s * (np.arange(r)[None, :] < rk_rv[si][:, None])   # dropped components
            dst[b, g, :m] = to_storage(_span_means(U, s, Vt, lens), dt)

    pairs = [(b, g) for b in range(B) for g in range(Hkv)]
    nthreads = threads if threads is not None else min(16, os.cpu_count() or 1)
    if nthreads > 1 and len(pairs) > 1:
        with ThreadPoolExecutor(nthreads) as ex:
            list(ex.map(work, pairs))
    else:
        for bg in pairs:
            work(bg)

    return Case(spec=spec, layer=layer, variant=variant, q=q_st, anchor_k=anchor_k,
                anchor_v=anchor_v, n_anchors=n_anch, sum_k=sum_k, sum_v=sum_v,
                n_spans=n_spans, span_len=span_len, span_logsize=span_logsize,
                factors=arena, block_off=block_off, needles=needles, block_rank=block_rank)


def with_top_k(case: Case, k: int) -> Case:
    """The same stored cache with a different top-k."""
    return replace(case, spec=replace(case.spec, top_k=k))


def case_from_factors(q, anchor_k, anchor_v, span_factors, *, dtype: str, top_k: int,
                      sum_k=None, sum_v=None) -> Case:
    """Pack caller-given float64 arrays into a stored cache.

    q: [B][Hq][d]; anchor_k/anchor_v: per sequence b an array [Hkv][A_b][d];
    span_factors: per sequence b a list (over spans S) of per-KV-head lists of
    dicts with keys UK [L][r], sK [r], VtK [r][d], UV, sV, VtV (all spans of a
    sequence share L across heads; r is common).  Summaries are the span means
    of the stored factors unless sum_k / sum_v ([B][Hkv][M][d]) are given.
    """
    q = np.asarray(q, dtype=np.float64)
    B, Hq, d = q.shape
    Hkv = np.asarray(anchor_k[0]).shape[0] if B else 1
    n_anch = np.array([np.asarray(a).shape[1] for a in anchor_k], dtype=np.int32)
    n_spans = np.array([len(sf) for sf in span_factors], dtype=np.int32)
    A_max = max(int(n_anch.max()) if B else 0, 1)
    M_max = max(int(n_spans.max()) if B else 0, 1)
    r = None
    for sf in span_factors:
        for per_head in sf:
            r = per_head[0]["UK"].shape[1]
            break
        if r is not None:
            break
    r = r or 8
    st_t = _np_storage_type(dtype)
    e = elem_bytes(dtype)
    spec = CaseSpec("packed", batch=B, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, rank=r,
                    top_k=top_k, context=0, n_prefix_anchors=0, window=0,
                    span_dist="uniform", span_min=1, span_max=1, dtype=dtype,
                    factor_kind="gaussian")
    span_len = np.zeros((B, M_max), dtype=np.int32)
    for b, sf in enumerate(span_factors):
        for S, per_head in enumerate(sf):
            span_len[b, S] = per_head[0]["UK"].shape[0]
    span_logsize = np.zeros((B, M_max))
    nz = span_len > 0
    span_logsize[nz] = np.log(span_len[nz].astype(np.float64))
    block_off = np.zeros((B, Hkv, M_max), dtype=np.int64)
    total = 0
    for b in range(B):
        for g in range(Hkv):
            for S in range(int(n_spans[b])):
                block_off[b, g, S] = total
                total += block_bytes(int(span_len[b, S]), r, d, dtype)
    arena = np.zeros(max(total, 256), dtype=np.uint8)
    arena_e = arena.view(st_t)
    ak = np.zeros((B, Hkv, A_max, d), dtype=st_t)
    av = np.zeros((B, Hkv, A_max, d), dtype=st_t)
    sk = np.zeros((B, Hkv, M_max, d), dtype=st_t)
    sv = np.zeros((B, Hkv, M_max, d), dtype=st_t)
    for b in range(B):
        A = int(n_anch[b])
        ak[b, :, :A] = to_storage(np.asarray(anchor_k[b], np.float64), dtype)
        av[b, :, :A] = to_storage(np.asarray(anchor_v[b], np.float64), dtype)
        for g in range(Hkv):
            m = int(n_spans[b])
            if m == 0:
                continue
            lens = [int(span_len[b, S]) for S in range(m)]
            fac_st = {}
            for side in ("K", "V"):
                U = np.concatenate([span_factors[b][S][g]["U" + side] for S in range(m)], axis=0)
                s = np.stack([span_factors[b][S][g]["s" + side] for S in range(m)])
                Vt = np.stack([span_factors[b][S][g]["Vt" + side] for S in range(m)])
                fac_st[side] = [to_storage(U, dtype), to_storage(s, dtype), to_storage(Vt, dtype)]
            _write_pair(spec, arena_e, block_off[b, g, :m] // e, lens, fac_st)
            for side, dst, given in (("K", sk, sum_k), ("V", sv, sum_v)):
                if given is not None:
                    dst[b, g, :m] = to_storage(np.asarray(given)[b, g, :m], dtype)
                else:
                    U, s, Vt = (from_storage(x, dtype) for x in fac_st[side])
                    dst[b, g, :m] = to_storage(_span_means(U, s, Vt, lens), dtype)
    case = Case(spec=spec, layer=0, variant="L", q=to_storage(q, dtype), anchor_k=ak,
                anchor_v=av, n_anchors=n_anch, sum_k=sk, sum_v=sv, n_spans=n_spans,
                span_len=span_len, span_logsize=span_logsize, factors=arena,
                block_off=block_off)
    return case


# ---------------------------------------------------------------------------
# inputs of the learned routing rule
# ---------------------------------------------------------------------------

NO_BUDGET = 1 << 62


@dataclass
class Gate:
    """Stored inputs of the learned selection rule for one layer.

    proj       [Hq][d'][d]        routing projection W of each query head (storage type)
    sum_route  [B][Hq][M_max][d'] normalised projected span summaries (storage type)
    thresholds [Hq] float64       zoom thresholds as pre-sigmoid values, ln(tau / (1 - tau))
    tau        [Hq] float64       the same thresholds as probabilities
    budget_tokens                 expanded tokens allowed per (sequence, KV head)
    """
    route_dim: int
    proj: np.ndarray
    sum_route: np.ndarray
    thresholds: np.ndarray
    tau: np.ndarray
    budget_tokens: int


def make_gate(case: Case, route_dim: int = 32, tau="permissive", budget_tokens: int = NO_BUDGET,
              proj_f64: np.ndarray | None = None) -> Gate:
    """Random stand-ins for the trained routing parameters of a case.

    The trained projections are not available: W[h] has i.i.d. normal entries of
    variance 1/d', so that (W q) . (W k) estimates q . k.  The routing summary of
    span S for head h is W[h] k_bar_S normalised, with k_bar_S the stored mean
    key of the span (with uniform token weights the weighted projected mean is the
    projection of the mean).  tau: "permissive" (0.05 for every head, the
    initialisation the paper trains from), a float or an array of per-head
    probabilities, or "spread": per-head thresholds ln(L_h) with L_h drawn
    log-uniformly from the span-length range, so that some spans of every
    length class fall on either side.  proj_f64 replaces the random W (its
    values are rounded to storage).
    """
    s = case.spec
    B, Hq, Hkv, d = s.batch, s.n_q_heads, s.n_kv_heads, s.head_dim
    G = Hq // Hkv
    dt = s.dtype
    dr = int(route_dim)
    vkey = (s.seed, VARIANTS[case.variant], case.layer)
    if proj_f64 is None:
        w64 = np.stack([normals(stream_key(*vkey, ST_PROJ, h), dr * d).reshape(dr, d)
                        for h in range(Hq)]) / math.sqrt(dr)
    else:
        w64 = np.asarray(proj_f64, dtype=np.float64).reshape(Hq, dr, d)
    proj = to_storage(w64, dt)
    wdec = from_storage(proj, dt)
    kbar = from_storage(case.sum_k, dt)
    M = case.sum_k.shape[2]
    sr = np.zeros((B, Hq, M, dr), dtype=np.float64)
    for b in range(B):
        m = int(case.n_spans[b])
        for h in range(Hq):
            x = kbar[b, h // G, :m] @ wdec[h].T
            nrm = np.sqrt((x * x).sum(axis=1))
            nz = nrm > 0
            sr[b, h, :m][nz] = x[nz] / nrm[nz, None]
    if isinstance(tau, str) and tau == "spread":
        u = uniforms(stream_key(*vkey, ST_TAU), Hq)
        lo, hi = math.log(max(s.span_min, 1)), math.log(max(s.span_max, 1) + 1)
        thr = lo + u * (hi - lo)
        taus = 1.0 / (1.0 + np.exp(-thr))
    else:
        taus = np.full(Hq, 0.05) if (isinstance(tau, str) and tau == "permissive") else \
            np.broadcast_to(np.asarray(tau, dtype=np.float64), (Hq,)).copy()
        thr = np.array([math.log(t / (1.0 - t)) for t in taus])
    return Gate(route_dim=dr, proj=proj, sum_route=to_storage(sr, dt), thresholds=thr,
                tau=taus, budget_tokens=int(budget_tokens))


# ---------------------------------------------------------------------------
# prefill inputs: token keys/values and surprisal (for the cache builder)
# ---------------------------------------------------------------------------

ST_SURP, ST_KTOK, ST_VTOK, ST_SPIKE, ST_OMEGA = 15, 16, 17, 18, 19


@dataclass
class Prefill:
    """Token-level inputs of the prefill-side builder for one layer.

    keys/values [B][Hkv][N_max][d] (storage type), surprisal [B][N_max] float32,
    n_tokens [B] int32, omega [d][l] float32 (the random test matrix of the
    randomized SVD, drawn here and passed in)."""
    keys: np.ndarray
    values: np.ndarray
    surprisal: np.ndarray
    n_tokens: np.ndarray
    omega: np.ndarray
    dtype: str
    true_starts: list = field(default_factory=list)


def make_prefill(batch: int, n_kv_heads: int, head_dim: int, n_tokens, dtype: str = "bf16",
                 spike_every: int = 150, true_rank: int = 24, noise: float = 0.02, sketch: int = 40,
                 seed: int = 0) -> Prefill:
    """Synthetic prefill of `batch` sequences.

    Surprisal: a background of 1 + 0.05 (sum of four Exp(1) draws - 4) with spikes of +8
    at roughly one position in `spike_every`, so that the mu + alpha sigma rule finds
    sparse boundaries.  Keys and values: inside each stretch between spikes,
    a random rank-`true_rank` matrix plus Gaussian noise of relative size `noise`, scaled
    by 1/sqrt(d) -- compressible spans, as the paper expects of coherent text."""
    d = head_dim
    n_tok = np.broadcast_to(np.asarray(n_tokens, dtype=np.int64), (batch,)).copy()
    N = max(int(n_tok.max()), 1)
    st = _np_storage_type(dtype)
    K = np.zeros((batch, n_kv_heads, N, d), dtype=st)
    V = np.zeros((batch, n_kv_heads, N, d), dtype=st)
    H = np.zeros((batch, N), dtype=np.float32)
    starts_all = []
    for b in range(batch):
        n = int(n_tok[b])
        e = uniforms(stream_key(seed, ST_SURP, b), 4 * n).reshape(4, n)
        h = 1.0 + 0.05 * ((-np.log1p(-e)).sum(axis=0) - 4.0)
        u = uniforms(stream_key(seed, ST_SPIKE, b), n)
        spike = u < 1.0 / spike_every
        h = h + 8.0 * spike
        H[b, :n] = h.astype(np.float32)
        starts = [0] + [int(t) for t in np.flatnonzero(spike)] + [n]
        starts_all.append(starts)
        for g in range(n_kv_heads):
            for side, arr, sk in (("K", K, ST_KTOK), ("V", V, ST_VTOK)):
                rows = np.zeros((n, d))
                for j in range(len(starts) - 1):
                    s0, s1 = starts[j], starts[j + 1]
                    L = s1 - s0
                    if L <= 0:
                        continue
                    key = stream_key(seed, sk, b, g, j)
                    z = normals(key, L * true_rank).reshape(L, true_rank)
                    A = normals(key + 1, true_rank * d).reshape(true_rank, d)
                    eps = normals(key + 2, L * d).reshape(L, d)
                    rows[s0:s1] = (z @ A / math.sqrt(true_rank) + noise * eps) / math.sqrt(d)
                arr[b, g, :n] = to_storage(rows, dtype)
    omega = normals(stream_key(seed, ST_OMEGA), d * sketch).reshape(d, sketch).astype(np.float32)
    return Prefill(keys=K, values=V, surprisal=H, n_tokens=n_tok.astype(np.int32), omega=omega, dtype=dtype,
                   true_starts=starts_all)
