"""Seeded synthetic Q/K/V for one attention layer with FlexPrefill-style structure.

The paper measures on real long-context prompts run through real models; neither
is available here, so every workload is a seeded synthetic layer with the head
counts, head dimension and sequence lengths of the models the paper evaluates
(Llama-3.1-8B, GLM-4-9B, Qwen2-7B shaped), and with the two kinds of attention
structure the paper describes in Section 2 ("Attention Sparse Patterns Exhibit
Variability"):

* vertical-slash heads: an attention sink at key 0, a handful of "vertical"
  keys that every query attends to, and a strong main diagonal;
* query-specific heads: keys grouped into contiguous clusters (random
  centroids), each query block attending to one to three centroids.

Construction (per sequence, per KV group g):

1. Base Q, K, V ~ N(0, 1) in float32, then rotary position embedding with
   theta = 1e4 (rotate-half pairing (k, k + d/2), position = index within the
   sequence) on Q and K.
2. A random orthonormal "structure" basis U_g (d x r) is drawn; base Q and K
   are projected out of span(U_g), so injected logit boosts are exact.  The
   first column u is the sink/vertical direction, the others hold centroids.
3. Vertical-slash heads: every query gets + alpha*u; key 0 gets
   + (beta_s*sqrt(d)/alpha)*u and each vertical key + (beta_v*sqrt(d)/alpha)*u,
   so their logits rise by exactly beta_s / beta_v.  Query i also gets
   + beta_d*sqrt(d)*k_i^perp/|k_i^perp|^2 (its own key direction), which raises
   the diagonal logit by exactly beta_d.
4. Query-specific heads: keys are cut into block-aligned segments of 1..4
   blocks, each with a random centroid c (unit vector in span(U_g[:,1:]));
   keys get + (beta_c*sqrt(d)/alpha_c)*c, and the queries of each query block
   get + alpha_c * (sum of 1..3 distinct random centroids).
5. The boosts are calibrated from target last-block attention fractions
   (sink, verticals, diagonal, background noise) using the log-normal estimate
   of the noise partition function, n*exp(sigma^2/2).

Everything is float32 and then rounded to bf16 (round to nearest even); the
device path and the oracle both consume exactly those bf16 values.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

ROPE_THETA = 1.0e4
ALPHA = 2.0          # query amplitude along the sink/vertical direction
ALPHA_C = 2.0        # query amplitude along each attended centroid
BETA_C = 7.0         # logit boost of an attended cluster
N_CENTROIDS = 64
# Target fractions of the last query block's attention mass (vertical-slash heads).
F_SINK, F_VERT, F_DIAG, F_NOISE = 0.45, 0.25, 0.28, 0.02

TENSOR_Q, TENSOR_K, TENSOR_V, TENSOR_STRUCT = 0, 1, 2, 3


@dataclass(frozen=True)
class LayerSpec:
    """Shape and structure of one synthetic attention layer."""
    name: str
    seqlens: tuple
    hq: int
    hkv: int
    d: int
    block: int
    head_kinds: tuple          # per query head: "vs" or "qa"
    n_vertical: int
    gamma: float
    tau: float
    min_budget: int            # minimum key blocks per query-block row
    seed: int
    gammas: tuple = field(default=())   # optional sweep

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seqlens))

    @property
    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seqlens)]).astype(np.int32)

    def with_seqlens(self, seqlens, name=None) -> "LayerSpec":
        return LayerSpec(name or self.name, tuple(int(s) for s in seqlens), self.hq, self.hkv,
                         self.d, self.block, self.head_kinds, self.n_vertical, self.gamma,
                         self.tau, self.min_budget, self.seed, self.gammas)

    def with_params(self, **kw) -> "LayerSpec":
        fields = dict(name=self.name, seqlens=self.seqlens, hq=self.hq, hkv=self.hkv, d=self.d,
                      block=self.block, head_kinds=self.head_kinds, n_vertical=self.n_vertical,
                      gamma=self.gamma, tau=self.tau, min_budget=self.min_budget,
                      seed=self.seed, gammas=self.gammas)
        fields.update(kw)
        return LayerSpec(**fields)


def _kinds(hq, rule):
    return tuple(rule(h) for h in range(hq))


def _even_vs(h):
    return "vs" if h % 2 == 0 else "qa"


SPECS = {
    # Tiny causal prefill: 2 query heads, 2 KV heads, d = 64, n = 2048, both vertical-slash.
    "tiny": LayerSpec("tiny-2h-d64-n2048", (2048,), 2, 2, 64, 128, ("vs", "vs"), 8,
                      0.9, 0.1, 1, 20250228 + 1),
    # Llama-3-8B-shaped layer at 32k: 32 q heads, 8 KV heads, d = 128, mixed heads.
    "llama32k": LayerSpec("llama3-8b-layer-n32768", (32768,), 32, 8, 128, 128,
                          _kinds(32, _even_vs), 16, 0.9, 0.1, 8, 20250228 + 2),
    # Same layer at 128k, gamma 0.95: the headline long-context case.
    "llama128k": LayerSpec("llama3-8b-layer-n131072", (131072,), 32, 8, 128, 128,
                           _kinds(32, _even_vs), 16, 0.95, 0.1, 8, 20250228 + 3),
    # GLM-4-9B-shaped layer: 32 q heads, 2 KV heads (GQA 16:1), 25% vertical-slash heads.
    "glm64k": LayerSpec("glm4-9b-layer-n65536", (65536,), 32, 2, 128, 128,
                        _kinds(32, lambda h: "vs" if h % 4 == 0 else "qa"), 16, 0.9, 0.2, 8,
                        20250228 + 4),
    # Qwen2-7B-shaped layer, 4 packed sequences of 16k..128k, 28 q heads, 4 KV heads.
    "qwen_varlen": LayerSpec("qwen2-7b-layer-varlen-245760", (16384, 32768, 65536, 131072), 28, 4,
                             128, 128, _kinds(28, _even_vs), 16, 0.9, 0.1, 8, 20250228 + 5,
                             gammas=(0.85, 0.9, 0.95)),
}


# ----------------------------------------------------------------------------------------------
# bf16 rounding (round to nearest even), the only precision conversion inputs go through.

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("bf16_bits: non-finite input")
    u = x.view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    flat_u, flat_o = u.reshape(-1), out.reshape(-1)
    step = 1 << 24
    for s in range(0, flat_u.size, step):
        c = flat_u[s:s + step]
        flat_o[s:s + step] = ((c + np.uint32(0x7FFF) + ((c >> np.uint32(16)) & np.uint32(1)))
                              >> np.uint32(16)).astype(np.uint16)
    return out


def bf16_bits_to_float(bits: np.ndarray) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    return bf16_bits_to_float(bf16_bits(x))


# ----------------------------------------------------------------------------------------------

def _rng(seed, seq, tensor_id, head):
    return np.random.default_rng(np.random.SeedSequence([int(seed), int(seq), int(tensor_id),
                                                         int(head)]))


class _Rope:
    """Cached cos/sin tables for rotate-half rotary embedding."""

    def __init__(self):
        self._cache = {}

    def __call__(self, x: np.ndarray) -> np.ndarray:
        n, d = x.shape
        key = (n, d)
        if key not in self._cache:
            half = d // 2
            inv = ROPE_THETA ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
            ang = np.arange(n, dtype=np.float64)[:, None] * inv[None, :]
            self._cache = {key: (np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32))}
        c, s = self._cache[key]
        half = d // 2
        x1, x2 = x[:, :half], x[:, half:]
        out = np.empty_like(x)
        out[:, :half] = x1 * c - x2 * s
        out[:, half:] = x1 * s + x2 * c
        return out


def structure_rank(d: int) -> int:
    return 8 if d <= 64 else 24


def vs_boosts(n: int, d: int, n_vertical: int):
    """Logit boosts (sink, vertical, diagonal) from the target mass fractions.

    Background logits q.k/sqrt(d) are ~N(0, s2) with s2 = (d-r)/d + beta_d^2/(d-r)
    (the second term is the cross talk of the diagonal injection).  The sink, the
    verticals and the background keys carry that noise, so each contributes about
    exp(beta + s2/2); the diagonal logit only carries the (d-r)/d part.  The noise
    partition function over n keys is about n*exp(s2/2).  Solved by fixed-point
    iteration on beta_d.
    """
    r = structure_rank(d)
    s0 = (d - r) / d
    beta_d = 10.0
    for _ in range(50):
        s2 = s0 + beta_d ** 2 / (d - r)
        z = n * math.exp(s2 / 2.0) / F_NOISE
        beta_d = math.log(F_DIAG * z) - s0 / 2.0
    beta_s = math.log(F_SINK * z) - s2 / 2.0
    beta_v = math.log(F_VERT * z / max(n_vertical, 1)) - s2 / 2.0
    return beta_s, beta_v, beta_d


@dataclass
class Layer:
    spec: LayerSpec
    q: np.ndarray            # [T, Hq, d] float32, bf16-representable
    k: np.ndarray            # [T, Hkv, d]
    v: np.ndarray            # [T, Hkv, d]
    cu_seqlens: np.ndarray   # [B+1] int32
    verticals: list          # per sequence: sorted vertical key positions (structure record)


def _orthonormal(rng, d, r):
    a = rng.standard_normal((d, r))
    qm, _ = np.linalg.qr(a)
    return qm.astype(np.float32)


def make_layer(spec: LayerSpec, heads=None, threads: int = 8) -> Layer:
    """Build the seeded layer.  `heads` optionally restricts which query heads are filled
    (the others stay zero) so that partial-head tests stay cheap.  KV groups are built in
    parallel threads; every draw comes from its own (seed, sequence, tensor, head) stream,
    so the result does not depend on the thread count."""
    from concurrent.futures import ThreadPoolExecutor

    d = spec.d
    T = spec.total_tokens
    q = np.zeros((T, spec.hq, d), dtype=np.float32)
    k = np.zeros((T, spec.hkv, d), dtype=np.float32)
    v = np.zeros((T, spec.hkv, d), dtype=np.float32)
    cu = spec.cu_seqlens
    head_set = set(range(spec.hq)) if heads is None else set(int(h) for h in heads)
    verticals = [[None] * spec.hkv for _ in spec.seqlens]
    tasks = [(s, g) for s in range(len(spec.seqlens)) for g in range(spec.hkv)]

    def run(task):
        s, g = task
        verticals[s][g] = _make_group(spec, s, g, int(cu[s]), head_set, q, k, v)

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(run, tasks))
    return Layer(spec, q, k, v, cu.copy(), verticals)


def _make_group(spec, s, g, t0, head_set, q, k, v):
    """Fill K, V of KV group g and the Q of its query heads for sequence s (rounded to
    bf16 in place).  Returns the vertical key positions."""
    d, b = spec.d, spec.block
    n = spec.seqlens[s]
    G = spec.hq // spec.hkv
    r = structure_rank(d)
    rope = _Rope()
    beta_s, beta_v, beta_d = vs_boosts(n, d, spec.n_vertical)
    group = range(g * G, (g + 1) * G)
    kinds = [spec.head_kinds[h] for h in group]
    srng = _rng(spec.seed, s, TENSOR_STRUCT, g)
    U = _orthonormal(srng, d, r)
    u = U[:, 0]
    cen = srng.standard_normal((N_CENTROIDS, r - 1)).astype(np.float32)
    cen /= np.linalg.norm(cen, axis=1, keepdims=True)
    cen = cen @ U[:, 1:].T                       # [C, d] unit vectors in span(U[:,1:])

    kg = rope(_rng(spec.seed, s, TENSOR_K, g).standard_normal((n, d), dtype=np.float32))
    kg -= (kg @ U) @ U.T
    k_perp = kg.copy()
    # vertical positions: distinct, uniform in [1, n - b) (none for sequences that short)
    hi = n - b
    nv = min(spec.n_vertical, hi - 1) if hi > 1 else 0
    verts = np.sort(srng.choice(np.arange(1, hi), size=nv, replace=False)) if nv > 0 \
        else np.zeros(0, dtype=np.int64)
    if "vs" in kinds:
        kg[0] += (beta_s * math.sqrt(d) / ALPHA) * u
        for vj in verts:
            kg[vj] += (beta_v * math.sqrt(d) / ALPHA) * u
    # query-specific clusters: block-aligned key segments of 1..4 blocks
    if "qa" in kinds:
        nb = -(-n // b)
        seg_centroid = np.empty(nb, dtype=np.int64)
        J = 0
        while J < nb:
            L = int(srng.integers(1, 5))
            seg_centroid[J:J + L] = int(srng.integers(0, N_CENTROIDS))
            J += L
        boost = (BETA_C * math.sqrt(d) / ALPHA_C)
        kg += boost * cen[np.repeat(seg_centroid, b)[:n]]
    k[t0:t0 + n, g] = round_to_bf16(kg)
    v[t0:t0 + n, g] = round_to_bf16(
        _rng(spec.seed, s, TENSOR_V, g).standard_normal((n, d), dtype=np.float32))

    kn2 = np.einsum("nd,nd->n", k_perp, k_perp).astype(np.float32)
    for h in group:
        if h not in head_set:
            continue
        qh = rope(_rng(spec.seed, s, TENSOR_Q, h).standard_normal((n, d), dtype=np.float32))
        qh -= (qh @ U) @ U.T
        if spec.head_kinds[h] == "vs":
            qh += ALPHA * u[None, :]
            qh += (beta_d * math.sqrt(d) / kn2)[:, None] * k_perp
        else:
            # each query block attends to m in {1,2,3} distinct random centroids
            hrng = _rng(spec.seed, s, TENSOR_STRUCT, 1000 + h)
            nbq = -(-n // b)
            m = hrng.integers(1, 4, size=nbq)
            perm = np.argsort(hrng.random((nbq, N_CENTROIDS)), axis=1)
            w = np.zeros((nbq, N_CENTROIDS), dtype=np.float32)
            rows_i = np.arange(nbq)
            for t in range(3):
                w[rows_i[m > t], perm[m > t, t]] = 1.0
            qh += np.repeat(ALPHA_C * (w @ cen), b, axis=0)[:n]
        q[t0:t0 + n, h] = round_to_bf16(qh)
    return verts
