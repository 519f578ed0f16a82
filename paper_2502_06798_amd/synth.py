"""Seeded synthetic workloads for the prompt-to-cache matching step.

This module only draws random inputs and rounds them to their storage type.
None of the matching arithmetic (similarity, top-k, levels, assignment,
gather) lives here, so both the HIP path and the CPU reference consume the
same bytes without sharing any of the method's code.

The paper measures on DiffusionDB prompts replayed from a Twitter trace
(Evaluation section); neither the prompts nor the embedding model are
available, so clustered Gaussian embeddings stand in for prompt embeddings:

* cluster centres c ~ N(0, I_d);
* a cache entry of cluster j is normalise(c_j + sigma_e * z), z ~ N(0, I_d);
* a query is normalise(c_j + sigma_q * z) for a uniformly drawn cluster j,
  sigma_q fixed or drawn per query from U(lo, hi);
* all of this in float64, rounded to float32, then to the storage type
  (f16/bf16 by round-to-nearest-even, e4m3fn with a per-row float32 scale
  amax/448 and a clamp to +-448 before rounding);
* cached latents are uniform(-1, 1) rounded to f16.

Every stream is seeded from ``SeedSequence([2502, 6798, workload, stream,
chunk])`` with chunks of 65,536 rows, so generation is chunked and
independent of the device's memory size.  The same seed yields the same
bytes on the same device type; the CPU and GPU random generators differ, so
a GPU test generates on the GPU and copies to the host what the reference
needs.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np
import torch

CHUNK = 65536

# random streams
S_CENTRES, S_ENTRY_CLUSTER, S_ENTRY_NOISE = 0, 1, 2
S_QUERY_CLUSTER, S_QUERY_SIGMA, S_QUERY_NOISE = 3, 4, 5
S_LATENTS, S_HOT, S_QUEUE = 6, 7, 8

DTYPES = ("f32", "f16", "bf16", "e4m3")
ELEM_BYTES = {"f32": 4, "f16": 2, "bf16": 2, "e4m3": 1}
TORCH_DTYPE = {"f32": torch.float32, "f16": torch.float16,
               "bf16": torch.bfloat16, "e4m3": torch.float8_e4m3fn}

# similarity thresholds and skip counts of the quality table: a larger skip
# K needs a closer cached prompt.  Five levels (K = 5..25) and ten levels
# (K = 5..50 with thresholds 0.70 + 0.03 (l - 1)), written as float32.
THETA5 = tuple(float(np.float32(v)) for v in (0.75, 0.80, 0.85, 0.90, 0.95))
K5 = (5, 10, 15, 20, 25)
THETA10 = tuple(float(np.float32(0.70 + 0.03 * i)) for i in range(10))
K10 = tuple(5 * (i + 1) for i in range(10))


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and distribution of one synthetic matching workload."""
    wid: int                 # seed component
    name: str
    B: int                   # queries per batch
    N: int                   # cache entries
    d: int                   # embedding width
    dtype: str               # storage type of embeddings and queries
    k: int                   # neighbours returned per query
    clusters: int
    sigma_e: float
    sigma_q: Tuple[float, float]     # (lo, hi); lo == hi means constant
    theta: Tuple[float, ...]
    K: Tuple[int, ...]
    n_inst: int
    cap: int
    latent_shape: Optional[Tuple[int, int, int]]   # (C, H, W) of f16 latents
    hot: Optional[int] = None        # resident latent slots (None = all entries)

    @property
    def L(self) -> int:
        return len(self.theta)

    @property
    def latent_bytes(self) -> int:
        if self.latent_shape is None:
            return 0
        c, h, w = self.latent_shape
        return c * h * w * 2

    @property
    def n_slots(self) -> int:
        if self.latent_shape is None:
            return 0
        return self.hot if self.hot is not None else self.N

    def scaled(self, B=None, N=None, name=None, hot=None, latent_shape="keep"):
        """Same distribution at another size (for CPU tests)."""
        return dataclasses.replace(
            self, B=B or self.B, N=N or self.N, name=name or self.name,
            hot=self.hot if hot is None else hot,
            latent_shape=self.latent_shape if latent_shape == "keep" else latent_shape)


WORKLOADS = (
    Workload(1, "b16_n10k_d768_f32", 16, 10_000, 768, "f32", 5, 100, 0.3, (0.4, 0.4),
             THETA5, K5, 2, 8, (4, 64, 64)),
    Workload(2, "b256_n100k_d768_f16", 256, 100_000, 768, "f16", 10, 1_000, 0.3, (0.4, 0.4),
             THETA5, K5, 4, 64, (4, 64, 64)),
    Workload(3, "b1024_n1m_d768_bf16", 1_024, 1_000_000, 768, "bf16", 10, 10_000, 0.3, (0.4, 0.4),
             THETA5, K5, 8, 128, (4, 128, 128)),
    Workload(4, "b4096_n4m_d512_f16", 4_096, 4_000_000, 512, "f16", 16, 20_000, 0.3, (0.2, 0.8),
             THETA10, K10, 16, 256, None),
    Workload(5, "b16384_n10m_d768_e4m3", 16_384, 10_000_000, 768, "e4m3", 32, 50_000, 0.3, (0.2, 0.8),
             THETA10, K10, 32, 512, (4, 128, 128), hot=512),
)
BY_NAME = {w.name: w for w in WORKLOADS}


def seed_of(wid: int, stream: int, chunk: int = 0) -> int:
    ss = np.random.SeedSequence([2502, 6798, wid, stream, chunk])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def _gen(device, wid, stream, chunk=0) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed_of(wid, stream, chunk))
    return g


def centres(w: Workload, device) -> torch.Tensor:
    """Cluster centres, float64, drawn in chunks of rows."""
    out = torch.empty((w.clusters, w.d), dtype=torch.float64, device=device)
    for c, r0 in enumerate(range(0, w.clusters, CHUNK)):
        r1 = min(w.clusters, r0 + CHUNK)
        out[r0:r1] = torch.randn((r1 - r0, w.d), dtype=torch.float64, device=device,
                                 generator=_gen(device, w.wid, S_CENTRES, c))
    return out


def to_storage(x32: torch.Tensor, dtype: str):
    """Round float32 rows to the storage type.

    Returns (stored rows, per-row float32 scale or None).  e4m3fn uses the
    scale amax/448 of each row and clamps to +-448 before the cast (the cast
    itself does not saturate).
    """
    if dtype == "f32":
        return x32.contiguous(), None
    if dtype in ("f16", "bf16"):
        return x32.to(TORCH_DTYPE[dtype]).contiguous(), None
    if dtype == "e4m3":
        amax = x32.abs().amax(dim=1)
        scale = (amax / 448.0).to(torch.float32)
        scale = torch.where(scale > 0, scale, torch.ones_like(scale))
        y = (x32 / scale[:, None]).clamp(-448.0, 448.0)
        return y.to(torch.float8_e4m3fn).contiguous(), scale.contiguous()
    raise ValueError(dtype)


def _rows(w: Workload, device, n_rows: int, s_cluster: int, s_noise: int,
          sigma_fn, out: torch.Tensor, scale_out: Optional[torch.Tensor], C: torch.Tensor):
    for c, r0 in enumerate(range(0, n_rows, CHUNK)):
        r1 = min(n_rows, r0 + CHUNK)
        n = r1 - r0
        cid = torch.randint(0, w.clusters, (n,), device=device,
                            generator=_gen(device, w.wid, s_cluster, c))
        z = torch.randn((n, w.d), dtype=torch.float64, device=device,
                        generator=_gen(device, w.wid, s_noise, c))
        sig = sigma_fn(c, n)
        x = C[cid] + sig * z
        x = x / torch.linalg.vector_norm(x, dim=1, keepdim=True)
        stored, scale = to_storage(x.to(torch.float32), w.dtype)
        out[r0:r1] = stored
        if scale_out is not None:
            scale_out[r0:r1] = scale


def entries(w: Workload, device, C: Optional[torch.Tensor] = None):
    """Cache-entry embeddings (N x d, storage type) and row scales (e4m3 only)."""
    C = centres(w, device) if C is None else C
    emb = torch.empty((w.N, w.d), dtype=TORCH_DTYPE[w.dtype], device=device)
    scale = torch.empty((w.N,), dtype=torch.float32, device=device) if w.dtype == "e4m3" else None
    _rows(w, device, w.N, S_ENTRY_CLUSTER, S_ENTRY_NOISE,
          lambda c, n: w.sigma_e, emb, scale, C)
    return emb, scale


def queries(w: Workload, device, C: Optional[torch.Tensor] = None, B: Optional[int] = None):
    """Query embeddings (B x d, storage type) and row scales (e4m3 only)."""
    C = centres(w, device) if C is None else C
    B = w.B if B is None else B
    q = torch.empty((B, w.d), dtype=TORCH_DTYPE[w.dtype], device=device)
    scale = torch.empty((B,), dtype=torch.float32, device=device) if w.dtype == "e4m3" else None
    lo, hi = w.sigma_q

    def sigma(c, n):
        if lo == hi:
            return lo
        u = torch.rand((n, 1), dtype=torch.float64, device=device,
                       generator=_gen(device, w.wid, S_QUERY_SIGMA, c))
        return lo + (hi - lo) * u

    _rows(w, device, B, S_QUERY_CLUSTER, S_QUERY_NOISE, sigma, q, scale, C)
    return q, scale


def latents(w: Workload, device, n_slots: Optional[int] = None) -> Optional[torch.Tensor]:
    """Latent pool as raw bytes (n_slots x latent_bytes, uint8), f16 uniform(-1, 1)."""
    if w.latent_shape is None:
        return None
    n_slots = w.n_slots if n_slots is None else n_slots
    per = w.latent_bytes // 2
    pool = torch.empty((n_slots, per), dtype=torch.float16, device=device)
    rows = max(1, (1 << 28) // (per * 4))       # ~256 MiB of float32 per chunk
    for c, r0 in enumerate(range(0, n_slots, rows)):
        r1 = min(n_slots, r0 + rows)
        u = torch.rand((r1 - r0, per), dtype=torch.float32, device=device,
                       generator=_gen(device, w.wid, S_LATENTS, c))
        pool[r0:r1] = (2.0 * u - 1.0).to(torch.float16)
    return pool.view(torch.uint8)


def slot_map(w: Workload, device) -> Optional[torch.Tensor]:
    """entry -> latent slot (int32, -1 = not resident), or None when every entry is resident."""
    if w.latent_shape is None or w.hot is None:
        return None
    g = _gen("cpu", w.wid, S_HOT)
    hot = torch.randperm(w.N, generator=g)[: w.hot]
    m = torch.full((w.N,), -1, dtype=torch.int32)
    m[hot] = torch.arange(w.hot, dtype=torch.int32)
    return m.to(device)


def instances(w: Workload):
    """Instance table (host numpy int32): level, capacity and queue length per instance.

    Instance i runs at level i mod (L + 1) (level 0 = no skip); queue
    lengths are seeded draws in [0, cap] and only order instances.
    """
    lvl = np.array([i % (w.L + 1) for i in range(w.n_inst)], dtype=np.int32)
    cap = np.full(w.n_inst, w.cap, dtype=np.int32)
    rng = np.random.default_rng(seed_of(w.wid, S_QUEUE))
    queue = rng.integers(0, w.cap + 1, size=w.n_inst).astype(np.int32)
    return lvl, cap, queue


def thresholds(w: Workload):
    """(theta float32[L], K int32[L]) as host numpy arrays."""
    return np.array(w.theta, dtype=np.float32), np.array(w.K, dtype=np.int32)


def host_view(t: Optional[torch.Tensor]):
    """Host numpy array of a tensor's stored elements (same bytes and element
    size: bfloat16 as int16, e4m3fn as uint8), or None."""
    if t is None:
        return None
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    if t.dtype == torch.float8_e4m3fn:
        return t.view(torch.uint8).numpy()
    return t.numpy()
