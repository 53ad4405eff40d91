"""Seeded synthetic inputs shaped like the paper's workloads.

This module holds none of the method's arithmetic: no quantizer, no distance
test, no scoring.  It only draws unit vectors, clustered members, planted
near-duplicates and arrival orders.  Both the oracle tests and the GPU path
take their inputs from here, so the two sides see identical bytes.

Everything is drawn with ``numpy.random.default_rng(seed)`` in float64 and cast
to float32 at the very end, with no re-normalisation after the cast (the
library receives the float32 rows exactly as a caller would hand them over).

Shapes follow the paper's workloads:
  * embeddings are unit-normalised, D = 768 (the encoder of the default
    configuration, Appendix "Implementation details", Table "config"), so the
    RMS coordinate is 1/sqrt(768) = 0.0361;
  * trajectories hold about 47 chunks (the 600-trajectory subset), the retrieval
    corpus holds 6,026 x 60 records (361,802 in total);
  * the quantizer microbenchmark is 2^26 fp32 values (Appendix "Measured
    hardware constants", Table "anchors").
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "unit_rows", "members", "near_dups", "cluster_sizes",
    "tiny_ingest", "subset_ingest", "raw_qeps", "corpus_retrieval",
    "online_store", "clustered", "near_threshold_pairs", "threshold_band_device", "dyadic_ties", "CONFIGS",
]


def _normalize(a: np.ndarray) -> np.ndarray:
    return a / np.linalg.norm(a, axis=-1, keepdims=True)


def unit_rows(rng: np.random.Generator, n: int, d: int) -> np.ndarray:
    """n rows normalize(N(0, I_d)), float64."""
    return _normalize(rng.standard_normal((n, d)))


def members(rng: np.random.Generator, mu: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Rows normalize(c*mu + sqrt(1-c^2)*u), u a random unit vector orthogonal
    to mu, so that each row has cosine c with its (unit) centre mu.  float64."""
    mu = np.atleast_2d(mu)
    g = rng.standard_normal(mu.shape)
    g -= np.sum(g * mu, axis=1, keepdims=True) * mu
    u = _normalize(g)
    c = np.asarray(c, dtype=np.float64).reshape(-1, 1)
    return _normalize(c * mu + np.sqrt(1.0 - c * c) * u)


def near_dups(rng: np.random.Generator, src: np.ndarray,
              lo: float = 0.96, hi: float = 0.995) -> np.ndarray:
    """A noisy copy of each source row at cosine ~U(lo, hi)."""
    c = rng.uniform(lo, hi, size=src.shape[0])
    return members(rng, src, c)


def cluster_sizes(total: int, n_clusters: int) -> np.ndarray:
    """Sizes as even as possible, larger clusters first (e.g. 27,986 over 600
    gives 386 x 47 + 214 x 46)."""
    base, extra = divmod(total, n_clusters)
    return np.array([base + 1] * extra + [base] * (n_clusters - extra), dtype=np.int64)


def clustered(rng: np.random.Generator, sizes, d: int,
              cmin: float = 0.80, cmax: float = 0.999, chunk: int = 1 << 16):
    """Members of Gaussian-centroid clusters at cosine ~U(cmin, cmax) to their
    centroid.  Returns (rows float64 in cluster order, centroids, labels)."""
    sizes = np.asarray(sizes, dtype=np.int64)
    cent = unit_rows(rng, sizes.size, d)
    labels = np.repeat(np.arange(sizes.size), sizes)
    out = np.empty((labels.size, d), dtype=np.float64)
    for s in range(0, labels.size, chunk):
        lab = labels[s:s + chunk]
        out[s:s + lab.size] = members(rng, cent[lab], rng.uniform(cmin, cmax, lab.size))
    return out, cent, labels


def _queries_near(rng, cent, nq, lo=0.5, hi=0.9):
    pick = rng.integers(0, cent.shape[0], nq)
    return members(rng, cent[pick], rng.uniform(lo, hi, nq))


def tiny_ingest(seed: int = 1, n: int = 4096, d: int = 768, dup_frac: float = 0.1,
                nq: int = 64):
    """4,096 unit Gaussian rows with 10% planted near-duplicates (noisy copies of
    an earlier-generated row at cosine 0.96-0.995), arrival order shuffled;
    64 random unit queries."""
    rng = np.random.default_rng(seed)
    n_dup = int(round(dup_frac * n))
    n_base = n - n_dup
    base = unit_rows(rng, n_base, d)
    src = rng.integers(0, n_base, n_dup)
    dups = near_dups(rng, base[src])
    x = np.concatenate([base, dups])
    source = np.concatenate([np.arange(n_base), src])     # generation source
    perm = rng.permutation(n)
    q = unit_rows(rng, nq, d)
    return dict(x=x[perm].astype(np.float32), source=source[perm],
                q=q.astype(np.float32), tau=0.95, eps=1e-3, k=10, batch=1024,
                name=f"tiny ingest n={n} D={d} dups={n_dup}")


def subset_ingest(seed: int = 2, n: int = 27986, n_traj: int = 600, d: int = 768,
                  nq: int = 1024):
    """Trajectories of ~47 chunks (600 clusters, member cosine ~U(0.80, 0.999)),
    trajectories in seeded random order, each one's chunks contiguous.  The
    queries (not part of the ingest) are drawn near random centroids at cosine
    ~U(0.5, 0.9), as in the retrieval workload."""
    rng = np.random.default_rng(seed)
    sizes = cluster_sizes(n, n_traj)
    rows, cent, labels = clustered(rng, sizes, d)
    order = rng.permutation(n_traj)
    starts = np.concatenate([[0], np.cumsum(sizes)[:-1]])
    idx = np.concatenate([np.arange(starts[t], starts[t] + sizes[t]) for t in order])
    q = _queries_near(rng, cent, nq)
    return dict(x=rows[idx].astype(np.float32), labels=labels[idx],
                q=q.astype(np.float32), tau=0.95, eps=1e-3, k=10, batch=1024,
                name=f"subset ingest n={n} D={d} trajectories={n_traj}")


def raw_qeps(seed: int = 3, log2n: int = 26):
    """2^26 fp32 values: first half N(0, 0.04^2), second half U(-1, 1)."""
    rng = np.random.default_rng(seed)
    n = 1 << log2n
    h = n // 2
    x = np.empty(n, dtype=np.float32)
    x[:h] = (0.04 * rng.standard_normal(h)).astype(np.float32)
    x[h:] = rng.uniform(-1.0, 1.0, n - h).astype(np.float32)
    return dict(x=x, eps_list=(1e-4, 1e-3, 1e-2), name=f"raw qeps n=2^{log2n}")


def corpus_retrieval(seed: int = 4, n: int = 361802, n_clusters: int = 6026,
                     d: int = 768, nq: int = 4096):
    """361,802 records in 6,026 clusters of ~60 (same cluster model), seeded
    store order; 4,096 queries near random centroids at cosine ~U(0.5, 0.9)."""
    rng = np.random.default_rng(seed)
    sizes = cluster_sizes(n, n_clusters)
    rows, cent, labels = clustered(rng, sizes, d)
    perm = rng.permutation(n)
    x = rows[perm].astype(np.float32)
    del rows
    q = _queries_near(rng, cent, nq)
    return dict(x=x, labels=labels[perm], q=q.astype(np.float32), eps=1e-3, k=10,
                name=f"corpus retrieval n={n} D={d} nq={nq}")


def online_store(seed: int = 5, n: int = 1 << 20, n_clusters: int = 16384,
                 d: int = 1024, dup_frac: float = 0.2, nq: int = 16384):
    """1,048,576 rows D=1024: 838,861 clustered base rows (16,384 clusters,
    cosine ~U(0.80, 0.999)) plus 209,715 planted near-duplicates of random base
    rows, arrival order a seeded permutation; 16,384 queries near random
    centroids, top-50."""
    rng = np.random.default_rng(seed)
    n_dup = int(round(dup_frac * n))
    n_base = n - n_dup
    sizes = cluster_sizes(n_base, n_clusters)
    base, cent, labels = clustered(rng, sizes, d)
    x = np.empty((n, d), dtype=np.float32)
    x[:n_base] = base
    src = rng.integers(0, n_base, n_dup)
    for s in range(0, n_dup, 1 << 16):
        x[n_base + s:n_base + min(n_dup, s + (1 << 16))] = \
            near_dups(rng, base[src[s:s + (1 << 16)]])
    del base
    perm = rng.permutation(n)
    x = x[perm]
    q = _queries_near(rng, cent, nq)
    return dict(x=x, q=q.astype(np.float32), tau=0.95, eps=1e-3, k=50, batch=4096,
                name=f"online store n={n} D={d} dups={n_dup}")


def online_store_device(seed: int = 5, device: str = "cuda", n: int = 1 << 20, n_clusters: int = 16384,
                        d: int = 1024, dup_frac: float = 0.2, nq: int = 16384):
    """The online-store recipe of `online_store` drawn on a device with torch's
    seeded generator (binary64 draws, float32 at the end), for tests at the
    full 1,048,576 x 1,024 size where drawing on the host takes minutes.  The
    values differ from `online_store` (another random stream); the recipe,
    shapes and distributions are the same.  Returns torch tensors on `device`."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    f64 = dict(device=device, dtype=torch.float64)

    def normalize(v):
        return v / torch.linalg.vector_norm(v, dim=1, keepdim=True)

    def members_dev(mu, c):
        gg = torch.randn(mu.shape, generator=g, **f64)
        gg -= (gg * mu).sum(dim=1, keepdim=True) * mu
        u = normalize(gg)
        c = c.reshape(-1, 1)
        return normalize(c * mu + torch.sqrt(1.0 - c * c) * u)

    def uniform(lo, hi, m):
        return lo + (hi - lo) * torch.rand(m, generator=g, **f64)

    n_dup = int(round(dup_frac * n))
    n_base = n - n_dup
    sizes = torch.from_numpy(cluster_sizes(n_base, n_clusters)).to(device)
    cent = normalize(torch.randn((n_clusters, d), generator=g, **f64))
    labels = torch.repeat_interleave(torch.arange(n_clusters, device=device), sizes)
    x = torch.empty((n, d), device=device, dtype=torch.float32)
    chunk = 1 << 16
    for s in range(0, n_base, chunk):
        lab = labels[s:s + chunk]
        x[s:s + lab.numel()] = members_dev(cent[lab], uniform(0.80, 0.999, lab.numel())).float()
    src = torch.randint(0, n_base, (n_dup,), generator=g, device=device)
    for s in range(0, n_dup, chunk):
        rows = x[src[s:s + chunk]].double()
        # the planted copies start from the float32 base rows
        x[n_base + s:n_base + s + rows.shape[0]] = members_dev(rows, uniform(0.96, 0.995, rows.shape[0])).float()
    perm = torch.randperm(n, generator=g, device=device)
    x = x[perm]
    pick = torch.randint(0, n_clusters, (nq,), generator=g, device=device)
    q = members_dev(cent[pick], uniform(0.5, 0.9, nq)).float()
    return dict(x=x, q=q, tau=0.95, eps=1e-3, k=50, batch=4096,
                name=f"online store (device draw) n={n} D={d} dups={n_dup}")


def threshold_band_device(seed: int = 21, device: str = "cuda", n: int = 200_000, d: int = 768,
                          tau: float = 0.95, spread: float = 3e-3):
    """n unit rows a_i (Gaussian; the second half heavy-tailed: coordinates
    scaled by 2^U(-6, 2) before normalising) and one row b_i per a_i at cosine
    tau + U(-spread, spread) to it, drawn on a device with torch's seeded
    generator (binary64 draws, float32 at the end).  Returns (a, b) as torch
    tensors on `device`."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    f64 = dict(device=device, dtype=torch.float64)

    def normalize(v):
        return v / torch.linalg.vector_norm(v, dim=1, keepdim=True)

    a = torch.randn((n, d), generator=g, **f64)
    h = n // 2
    a[h:] *= torch.exp2(-6.0 + 8.0 * torch.rand((n - h, d), generator=g, **f64))
    a = normalize(a)
    c = (tau + spread * (2.0 * torch.rand(n, generator=g, **f64) - 1.0)).reshape(-1, 1)
    gg = torch.randn((n, d), generator=g, **f64)
    gg -= (gg * a).sum(dim=1, keepdim=True) * a
    b = normalize(c * a + torch.sqrt(1.0 - c * c) * normalize(gg))
    return a.float(), b.float()


def near_threshold_pairs(rng: np.random.Generator, n_pairs: int, d: int, tau: float,
                         spread: float = 1e-7):
    """Pairs (a, b) of unit rows whose cosine is tau + U(-spread, spread), to
    drive decisions into the last bits of the threshold test."""
    a = unit_rows(rng, n_pairs, d)
    c = tau + rng.uniform(-spread, spread, n_pairs)
    b = members(rng, a, c)
    return a.astype(np.float32), b.astype(np.float32)


def dyadic_ties(rng: np.random.Generator, n_pairs: int, d: int):
    """Pairs planted exactly on the threshold tau = 0.9375 (delta^2 = 1/8):
    a is a random unit row rounded to the grid 2^-12 (exact in float32) and
    b = a + (e_i - e_j)/4, so sum (a - b)^2 = 1/16 + 1/16 exactly.  Returns
    (a, b, b_in, b_out, tau) where b_in / b_out move one coordinate of b by one
    float32 ulp towards / away from a."""
    a = np.round(unit_rows(rng, n_pairs, d) * 4096.0) / 4096.0
    i = rng.integers(0, d, n_pairs)
    j = (i + 1 + rng.integers(0, d - 1, n_pairs)) % d
    r = np.arange(n_pairs)
    b = a.copy()
    b[r, i] += 0.25
    b[r, j] -= 0.25
    a32, b32 = a.astype(np.float32), b.astype(np.float32)
    b_in, b_out = b32.copy(), b32.copy()
    b_in[r, i] = np.nextafter(b32[r, i], a32[r, i])
    b_out[r, i] = np.nextafter(b32[r, i], np.float32(np.inf) * np.sign(b32[r, i] - a32[r, i]))
    return a32, b32, b_in, b_out, 0.9375


CONFIGS = {
    "tiny": tiny_ingest,
    "subset": subset_ingest,
    "raw": raw_qeps,
    "corpus": corpus_retrieval,
    "online": online_store,
}
