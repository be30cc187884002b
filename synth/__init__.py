"""Seeded synthetic workloads for expert-map matching and prefetch selection.

This module only *draws inputs*: gate-probability maps, trajectory queries,
semantic embeddings, observed depths and layer ranges.  It holds none of the
arithmetic of the method itself (no cosine, no ranking, no thresholding), so
both the CPU oracle and the GPU path can take their inputs from here without
sharing any of the computation they are compared on.

Shapes follow the three models of Table 1 (Mixtral-8x7B: 32 layers x 8
experts, Qwen1.5-MoE: 24 x 60, Phi-3.5-MoE: 32 x 16).  The paper's own
workloads (LMSYS-Chat-1M / ShareGPT prompts run through those models) are not
available; clustered synthetic stores stand in for them:

* an expert map is ``softmax_row(Z_c + sigma * eps)`` per layer row, with
  cluster centroids ``Z_c ~ N(0, 1)^(L x E)`` and ``c ~ U{0..C-1}`` — a gate
  softmax as in the expert-map definition of Section 4.1;
* a trajectory query copies a stored map's logits (``log p``), adds
  ``(sigma / 2) * eps`` and re-applies the row softmax, then only its first
  ``depth`` layers count as observed (Section 4.2.2);
* a semantic embedding is ``x = mu_c + 0.3 * eps`` with ``mu_c ~ N(0, I_d)``,
  normalised to unit length and rounded to bf16 (Section 4.2.1 uses the
  embedding-layer output; its pooling is outside the matched quantity).

bf16 values are carried as ``uint16`` bit patterns produced by
round-to-nearest-even from float32.
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import hashlib
import os
from typing import Dict, Optional

import numpy as np

ROOT_SEED = 250205370

_STREAMS = (
    "map_centroids", "map_assign", "map_noise",
    "query_src", "query_noise", "depth",
    "emb_centroids", "emb_assign", "emb_noise",
    "qemb_assign", "qemb_noise",
    "new_assign", "new_map_noise", "new_emb_noise", "new_dup",
)

F32 = "f32"
BF16 = "bf16"


def rng(config_no: int, stream: str) -> np.random.Generator:
    """Independent PCG64 stream ``stream`` of workload ``config_no``."""
    ss = np.random.SeedSequence(ROOT_SEED, spawn_key=(int(config_no), _STREAMS.index(stream)))
    return np.random.Generator(np.random.PCG64(ss))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    # in-place uint32 steps with uint32 constants (the same values as the
    # plain expression, several times faster on large arrays)
    r = u >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    out = r.astype(np.uint16)
    mag = u & np.uint32(0x7FFFFFFF)
    nan = mag > np.uint32(0x7F800000)
    if nan.any():
        out[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
    return out


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def values_f32(arr: np.ndarray, dtype: str) -> np.ndarray:
    """The float32 values an array of ``dtype`` stands for (bf16 widened exactly)."""
    return bf16_to_f32(arr) if dtype == BF16 else np.asarray(arr, dtype=np.float32)


def _row_softmax_f32(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.float64)
    z -= z.max(axis=-1, keepdims=True)
    np.exp(z, out=z)
    z /= z.sum(axis=-1, keepdims=True)
    return z.astype(np.float32)


def _cast(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits(x) if dtype == BF16 else np.ascontiguousarray(x, dtype=np.float32)


@dataclasses.dataclass(frozen=True)
class Spec:
    """One synthetic workload: store, query batch and selection parameters."""
    config_no: int
    name: str
    n: int                      # stored maps
    L: int                      # MoE layers
    E: int                      # experts per layer (the paper's J)
    map_dtype: str
    map_centroids: int
    map_sigma: float
    d_emb: int = 0              # 0: no semantic embeddings
    emb_centroids: int = 0
    emb_sigma: float = 0.3
    B_traj: int = 0
    B_sem: int = 0
    depth_law: str = "uniform"  # "uniform": U{1..depth_max}; "geometric": min(Geom(p), depth_max)
    depth_max: int = 1
    depth_p: float = 0.15
    k: int = 1                  # matches kept per query
    blend: int = 0              # 0: use the top-1 map, 1: similarity-weighted top-k mean
    tau_mode: int = 0           # 0: fixed tau, 1: tau = clip(1 - score, 0, 1)
    tau: float = 0.9
    k_min: int = 1
    k_max: int = 8
    map_of_emb_mod: int = 0     # map centroid = embedding centroid mod this (paired stores)

    @property
    def B(self) -> int:
        return self.B_sem + self.B_traj

    def scaled(self, n: Optional[int] = None, B_traj: Optional[int] = None,
               B_sem: Optional[int] = None, **kw) -> "Spec":
        upd = dict(kw)
        if n is not None:
            upd["n"] = int(n)
        if B_traj is not None:
            upd["B_traj"] = int(B_traj)
        if B_sem is not None:
            upd["B_sem"] = int(B_sem)
        return dataclasses.replace(self, **upd)


def spec(config_no: int) -> Spec:
    """The five workloads at full size."""
    if config_no == 1:   # Mixtral-8x7B shape, tiny store
        return Spec(1, "mixtral_traj_n1k", n=1000, L=32, E=8, map_dtype=F32, map_centroids=16,
                    map_sigma=0.5, B_traj=8, depth_law="uniform", depth_max=31,
                    k=1, tau=0.9, k_min=1, k_max=4)
    if config_no == 2:   # Qwen1.5-MoE shape, trajectory matching
        return Spec(2, "qwen_traj_n50k_b64", n=50_000, L=24, E=60, map_dtype=F32, map_centroids=256,
                    map_sigma=0.7, B_traj=64, depth_law="uniform", depth_max=23,
                    k=1, tau=0.8, k_min=1, k_max=8)
    if config_no == 3:   # semantic matching, Mixtral-shaped maps paired with d=4096 embeddings
        return Spec(3, "semantic_d4096_n100k_b256", n=100_000, L=32, E=8, map_dtype=F32,
                    map_centroids=16, map_sigma=0.5, d_emb=4096, emb_centroids=512, emb_sigma=0.3,
                    B_sem=256, k=1, tau=0.9, k_min=1, k_max=8, map_of_emb_mod=16)
    if config_no == 4:   # Phi-3.5-MoE shape, decode-step trajectory matching, top-4 blend
        return Spec(4, "phi_traj_top4_n200k_b512", n=200_000, L=32, E=16, map_dtype=F32,
                    map_centroids=1024, map_sigma=0.6, B_traj=512, depth_law="geometric",
                    depth_max=31, depth_p=0.15, k=4, blend=1, tau=0.85, k_min=1, k_max=4)
    if config_no == 5:   # Qwen shape, bf16 store with d=2048 embeddings, mixed batch
        return Spec(5, "qwen_mixed_bf16_n1m_b1024", n=1_000_000, L=24, E=60, map_dtype=BF16,
                    map_centroids=256, map_sigma=0.7, d_emb=2048, emb_centroids=512, emb_sigma=0.3,
                    B_traj=512, B_sem=512, depth_law="uniform", depth_max=23,
                    k=1, tau=0.8, k_min=1, k_max=8, map_of_emb_mod=256)
    raise ValueError(f"no workload {config_no}")


_CHUNK = 16384


def _draw_depths(s: Spec) -> np.ndarray:
    g = rng(s.config_no, "depth")
    if s.depth_law == "uniform":
        d = g.integers(1, s.depth_max + 1, size=s.B_traj)
    elif s.depth_law == "geometric":
        d = np.minimum(g.geometric(s.depth_p, size=s.B_traj), s.depth_max)
    else:
        raise ValueError(s.depth_law)
    return d.astype(np.int32)


def _emb_centroids(s: Spec) -> np.ndarray:
    return rng(s.config_no, "emb_centroids").standard_normal((s.emb_centroids, s.d_emb), dtype=np.float32)


def _chunked(n: int, draw, finish) -> None:
    """For chunks [a, b) of n rows in order: draw(a, b) in this thread (the
    random streams are consumed in chunk order), finish(a, b, drawn) on a
    worker thread (elementwise NumPy work, so the result does not depend on
    the threads)."""
    workers = max(1, min(8, os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        pending = []
        for a in range(0, n, _CHUNK):
            b = min(a + _CHUNK, n)
            pending.append(ex.submit(finish, a, b, draw(a, b)))
            if len(pending) >= workers:
                pending.pop(0).result()
        for f in pending:
            f.result()


def _draw_embeddings(s: Spec, mu: np.ndarray, assign: np.ndarray, noise: np.random.Generator) -> np.ndarray:
    out = np.empty((assign.shape[0], s.d_emb), dtype=np.uint16)

    def draw(a, b):
        return noise.standard_normal((b - a, s.d_emb), dtype=np.float32)

    def finish(a, b, eps):
        x = mu[assign[a:b]] + np.float32(s.emb_sigma) * eps
        x = x.astype(np.float64)
        x /= np.linalg.norm(x, axis=1, keepdims=True)
        out[a:b] = bf16_bits(x.astype(np.float32))

    _chunked(assign.shape[0], draw, finish)
    return out


def generate(s: Spec) -> Dict[str, np.ndarray]:
    """Draw every array of workload ``s``.

    Returns a dict with
      maps    [n][L][E]  float32, or uint16 bf16 bits when ``map_dtype == "bf16"``
      embs    [n][d_emb] uint16 bf16 bits (absent when d_emb == 0)
      q_traj  [B_traj][L][E] same dtype as maps
      depth   [B_traj] int32 in [1, depth_max]
      src     [B_traj] int32: stored map each trajectory query was drawn from
      q_sem   [B_sem][d_emb] uint16 bf16 bits (absent when B_sem == 0)
      lb, le  [B] int32: layer range [lb, le) to select for, semantic queries first
    """
    n, L, E = s.n, s.L, s.E
    out: Dict[str, np.ndarray] = {}
    Zc = rng(s.config_no, "map_centroids").standard_normal((s.map_centroids, L, E), dtype=np.float32)
    emb_assign = None
    if s.d_emb:
        mu = _emb_centroids(s)
        emb_assign = rng(s.config_no, "emb_assign").integers(0, s.emb_centroids, size=n)
        out["embs"] = _draw_embeddings(s, mu, emb_assign, rng(s.config_no, "emb_noise"))
    if emb_assign is not None and s.map_of_emb_mod:
        cent = emb_assign % s.map_of_emb_mod
    else:
        cent = rng(s.config_no, "map_assign").integers(0, s.map_centroids, size=n)
    maps = np.empty((n, L, E), dtype=np.uint16 if s.map_dtype == BF16 else np.float32)
    noise = rng(s.config_no, "map_noise")

    def draw(a, b):
        return noise.standard_normal((b - a, L, E), dtype=np.float32)

    def finish(a, b, eps):
        z = Zc[cent[a:b]] + np.float32(s.map_sigma) * eps
        maps[a:b] = _cast(_row_softmax_f32(z), s.map_dtype)

    _chunked(n, draw, finish)
    out["maps"] = maps

    lb = []
    le = []
    if s.B_sem:
        qa = rng(s.config_no, "qemb_assign").integers(0, s.emb_centroids, size=s.B_sem)
        out["q_sem"] = _draw_embeddings(s, mu, qa, rng(s.config_no, "qemb_noise"))
        lb += [0] * s.B_sem
        le += [L] * s.B_sem
    if s.B_traj:
        src = rng(s.config_no, "query_src").integers(0, n, size=s.B_traj).astype(np.int32)
        base = values_f32(maps[src], s.map_dtype).astype(np.float64)
        with np.errstate(divide="ignore"):
            logit = np.log(base)
        logit += (s.map_sigma / 2.0) * rng(s.config_no, "query_noise").standard_normal(base.shape)
        out["q_traj"] = _cast(_row_softmax_f32(logit), s.map_dtype)
        depth = _draw_depths(s)
        out["depth"] = depth
        out["src"] = src
        lb += list(depth)
        le += [L] * s.B_traj
    out["lb"] = np.asarray(lb, dtype=np.int32)
    out["le"] = np.asarray(le, dtype=np.int32)
    return out


def generate_new(s: Spec, m: int, stored: Dict[str, np.ndarray], dup_frac: float = 0.125) -> Dict[str, np.ndarray]:
    """A batch of ``m`` new iterations for a store drawn by ``generate(s)``.

    New maps and embeddings come from the same clusters as the stored ones
    (fresh noise streams); a fraction ``dup_frac`` of them are exact copies of
    randomly chosen stored iterations (repeated prompts).  Returns
      new_maps [m][L][E] (store dtype), new_embs [m][d_emb] bf16 bits (absent
      when d_emb == 0), dup_src [m] int32 (stored index copied, -1 if none).
    """
    L, E = s.L, s.E
    n = stored["maps"].shape[0]
    Zc = rng(s.config_no, "map_centroids").standard_normal((s.map_centroids, L, E), dtype=np.float32)
    g = rng(s.config_no, "new_assign")
    out: Dict[str, np.ndarray] = {}
    if s.d_emb:
        mu = _emb_centroids(s)
        ea = g.integers(0, s.emb_centroids, size=m)
        out["new_embs"] = _draw_embeddings(s, mu, ea, rng(s.config_no, "new_emb_noise"))
        cent = ea % s.map_of_emb_mod if s.map_of_emb_mod else g.integers(0, s.map_centroids, size=m)
    else:
        cent = g.integers(0, s.map_centroids, size=m)
    z = Zc[cent] + np.float32(s.map_sigma) * rng(s.config_no, "new_map_noise").standard_normal(
        (m, L, E), dtype=np.float32)
    out["new_maps"] = _cast(_row_softmax_f32(z), s.map_dtype)
    d = rng(s.config_no, "new_dup")
    dup = np.full(m, -1, dtype=np.int32)
    if n > 0:
        pick = d.random(m) < dup_frac
        dup[pick] = d.integers(0, n, size=int(pick.sum()))
        out["new_maps"][pick] = stored["maps"][dup[pick]]
        if s.d_emb:
            out["new_embs"][pick] = stored["embs"][dup[pick]]
    out["dup_src"] = dup
    return out


def digests(arrays: Dict[str, np.ndarray]) -> Dict[str, str]:
    """SHA-256 of every generated array (bytes in C order)."""
    return {k: hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest() for k, v in sorted(arrays.items())}
