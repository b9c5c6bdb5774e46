"""Seeded input synthesis (no method arithmetic).

Two families of inputs:

* ``tiny_case``: the small fp32 case (1 layer, batch 1, 4 query / 2 KV heads,
  head_dim 64, 512 cached rows, 16 decode steps).  Q, K, V ~ N(0, 1) from a
  PCG64 stream; in each KV group 8 randomly chosen cached keys are shifted by
  3 * qbar, where qbar = sqrt(D) * unit(mean of the run's queries of that
  group), so that attention is concentrated on a few heavy hitters.

* ``ZipfCache``: Llama-8B / Qwen-7B-shaped caches generated on the GPU with
  torch's seeded Philox generator.  Per (layer, sequence, KV head) a unit
  direction u is drawn; queries are z + sqrt(D) * u and keys z_j + beta_j * u
  with beta_j = -s_l * ln(rho_j), rho_j a random rank in [1, T_b]; values are
  N(0, 1).  Scaled logits are then about beta_j plus unit-scale noise, so the
  attention a layer pays a token follows a Zipf law of exponent s_l; the
  per-layer exponent profile sets how sparse each layer is (the paper's
  layerwise sparsity heatmaps show non-monotone profiles that drift in time).

Score vectors for the selection/compaction tests come from ``score_vector``.
"""
import math

import numpy as np

from .configs import CONFIGS


# ----------------------------------------------------------------------------
# Small host-side cases
# ----------------------------------------------------------------------------

def tiny_case(seed=1):
    """The small fp32 case.  Returns a dict of float32 numpy arrays:
    K0, V0 (B, H_KV, 512, D); q (steps, B, H_Q, D); k_new, v_new
    (steps, B, H_KV, D) and the heavy-hitter indices (H_KV, 8)."""
    cfg = CONFIGS[1]
    rng = np.random.Generator(np.random.PCG64(seed))
    B, HQ, HK, D, T = cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.prompt
    G = HQ // HK
    steps = cfg.decode_steps
    q = rng.standard_normal((steps, B, HQ, D)).astype(np.float32)
    K0 = rng.standard_normal((B, HK, T, D)).astype(np.float32)
    V0 = rng.standard_normal((B, HK, T, D)).astype(np.float32)
    k_new = rng.standard_normal((steps, B, HK, D)).astype(np.float32)
    v_new = rng.standard_normal((steps, B, HK, D)).astype(np.float32)
    heavy = np.zeros((HK, 8), dtype=np.int64)
    for b in range(B):
        for h in range(HK):
            qm = q[:, b, h * G:(h + 1) * G].reshape(-1, D).astype(np.float64).mean(axis=0)
            qbar = math.sqrt(D) * qm / np.linalg.norm(qm)
            idx = rng.choice(T, size=8, replace=False)
            heavy[h] = idx
            K0[b, h, idx] += (3.0 * qbar).astype(np.float32)
    return {"K0": K0, "V0": V0, "q": q, "k_new": k_new, "v_new": v_new, "heavy": heavy}


def random_segment(rng, n, D, G, scale_k=1.0):
    """One segment of N(0,1) keys/values and G queries (float32)."""
    q = rng.standard_normal((G, D)).astype(np.float32)
    K = (scale_k * rng.standard_normal((n, D))).astype(np.float32)
    V = rng.standard_normal((n, D)).astype(np.float32)
    return q, K, V


def to_bf16_values(x):
    """Round float32 values to the nearest bfloat16 (ties to even) and return
    them widened back to float32, so host arrays hold exactly what a bf16
    device buffer stores."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) & 0xFFFF
    nan = np.isnan(x)
    r = np.where(nan, (u >> 16) | 0x40, r)
    return (r.astype(np.uint32) << 16).view(np.float32).reshape(x.shape)


def score_vector(rng, n, kind="zipf"):
    """Non-negative float32 score vectors with the structure the selection
    sees: ``zipf`` (few large, long tail), ``ties`` (values from a small set),
    ``special`` (ties plus +0/-0, NaN and +inf), ``uniform`` (continuous)."""
    if kind == "uniform":
        return rng.random(n).astype(np.float32)
    if kind == "zipf":
        ranks = rng.integers(1, max(n, 2) + 1, size=n)
        s = ranks.astype(np.float64) ** (-1.2) * (1.0 + 0.05 * rng.random(n))
        return s.astype(np.float32)
    if kind == "ties":
        levels = np.array([0.0, 0.125, 0.25, 0.5, 1.0, 3.0], dtype=np.float32)
        return levels[rng.integers(0, len(levels), size=n)]
    if kind == "special":
        levels = np.array([0.0, -0.0, 0.25, 0.5, 2.0, np.inf, np.nan], dtype=np.float32)
        return levels[rng.integers(0, len(levels), size=n)]
    raise ValueError(kind)


# ----------------------------------------------------------------------------
# Device-side Zipf caches (torch on the GPU)
# ----------------------------------------------------------------------------

def _seed(*parts):
    h = 0x9E3779B97F4A7C15
    for p in parts:
        h = (h ^ (int(p) & 0xFFFFFFFFFFFFFFFF)) * 0x100000001B3 & 0xFFFFFFFFFFFFFFFF
    return h & 0x7FFFFFFFFFFFFFFF


class ZipfCache:
    """Generates the Zipf key-bias inputs of one workload on a torch device.

    Everything is a deterministic function of (config, seed, tensor, layer,
    sequence): ``lengths()`` the logical lengths T_b, ``exponents()`` the
    per-layer Zipf exponents s_l, ``segment(l, b, n)`` the first n cached rows
    of every KV head of (l, b), ``step(t, l)`` one decode step's q, k_new, v_new.
    """

    def __init__(self, cfg_id, seed=None, device="cuda"):
        import torch
        self.torch = torch
        self.cfg = CONFIGS[cfg_id]
        self.cfg_id = cfg_id
        self.seed = cfg_id if seed is None else seed
        self.device = device
        self.dtype = torch.bfloat16 if self.cfg.dtype == "bf16" else torch.float32

    def _gen(self, *tag):
        g = self.torch.Generator(device=self.device)
        g.manual_seed(_seed(self.seed, self.cfg_id, *tag))
        return g

    def lengths(self):
        """Logical lengths T_b (prompt or drawn cached length) per sequence."""
        cfg = self.cfg
        rng = np.random.Generator(np.random.PCG64(_seed(self.seed, self.cfg_id, 1)))
        if cfg.length_dist == "fixed":
            return np.full(cfg.batch, cfg.prompt, dtype=np.int64)
        lo, hi = cfg.length_range
        if cfg.length_dist == "uniform":
            return rng.integers(lo, hi + 1, size=cfg.batch).astype(np.int64)
        if cfg.length_dist == "loguniform":
            return np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), size=cfg.batch))).astype(np.int64)
        raise ValueError(cfg.length_dist)

    def exponents(self):
        """Per-layer Zipf exponents s_l."""
        cfg = self.cfg
        L = cfg.num_layers
        if cfg.zipf == "ucurve":
            return np.array([1.2 + 0.4 * math.cos(2 * math.pi * l / (L - 1)) for l in range(L)])
        rng = np.random.Generator(np.random.PCG64(_seed(self.seed, self.cfg_id, 2)))
        lo, hi = cfg.zipf_range
        return rng.uniform(lo, hi, size=L)

    def layer_weights(self):
        """Fixed per-layer budget shares f_l (mean 10%, range 2%-40%, a
        seeded permutation of layer order) and the layer sparsities
        S_l = 1 - f_l / max(f) that make density weights proportional to f_l."""
        L = self.cfg.num_layers
        rng = np.random.Generator(np.random.PCG64(_seed(self.seed, self.cfg_id, 3)))
        perm = rng.permutation(L)
        f = np.array([0.02 * 20.0 ** ((perm[l] / (L - 1)) ** 1.6) for l in range(L)])
        return f, (1.0 - f / f.max()).astype(np.float32)

    def _epochs(self):
        cfg = self.cfg
        if cfg.zipf == "drift" and cfg.epoch > 0:
            return max(1, -(-cfg.decode_steps // cfg.epoch))
        return 1

    def directions(self, l, b=None):
        """Orthonormal key directions u_e of layer l: shape (H_KV, E, D) for
        one sequence b, or (B, H_KV, E, D) for all sequences."""
        torch = self.torch
        cfg = self.cfg
        E = self._epochs()
        if not hasattr(self, "_dirs"):
            self._dirs = {}
        if l not in self._dirs:
            us = []
            for bb in range(cfg.batch):
                z = torch.randn((cfg.num_kv_heads, cfg.head_dim, E), generator=self._gen(10, l, bb),
                                device=self.device, dtype=torch.float32)
                qm, _ = torch.linalg.qr(z.cpu().double())  # small; LAPACK on the host
                us.append(qm.float().to(self.device).transpose(1, 2).contiguous())
            self._dirs[l] = torch.stack(us)
        return self._dirs[l] if b is None else self._dirs[l][b]

    def segment(self, l, b, n, T=None):
        """Cached rows [0, n) of every KV head of (l, b): K, V of shape
        (H_KV, n, D) in the storage dtype."""
        torch = self.torch
        cfg = self.cfg
        T = int(self.lengths()[b]) if T is None else T
        H, D = cfg.num_kv_heads, cfg.head_dim
        u = self.directions(l, b)
        s_l = float(self.exponents()[l])
        g = self._gen(11, l, b)
        K = torch.randn((H, n, D), generator=g, device=self.device, dtype=torch.float32)
        E = u.shape[1]
        for e in range(E):
            rho = torch.randint(1, max(T, 1) + 1, (H, n), generator=g, device=self.device).float()
            beta = -s_l * torch.log(rho)
            K += beta[:, :, None] * u[:, e][:, None, :]
        V = torch.randn((H, n, D), generator=self._gen(12, l, b), device=self.device, dtype=torch.float32)
        return K.to(self.dtype), V.to(self.dtype)

    def step(self, t, l, T=None):
        """q (B, H_Q, D), k_new and v_new (B, H_KV, D) for decode step t of
        layer l; T (B,) are the logical lengths before the step."""
        torch = self.torch
        cfg = self.cfg
        B, H, D, G = cfg.batch, cfg.num_kv_heads, cfg.head_dim, cfg.group
        Ts = torch.as_tensor(self.lengths() if T is None else np.asarray(T), device=self.device)
        e = (t // cfg.epoch) if (cfg.zipf == "drift" and cfg.epoch > 0) else 0
        g = self._gen(20, t, l)
        u = self.directions(l)                                   # (B, H, E, D)
        E = u.shape[2]
        q = torch.randn((B, H * G, D), generator=g, device=self.device, dtype=torch.float32)
        k = torch.randn((B, H, D), generator=g, device=self.device, dtype=torch.float32)
        v = torch.randn((B, H, D), generator=g, device=self.device, dtype=torch.float32)
        q += math.sqrt(D) * u[:, :, min(e, E - 1)].repeat_interleave(G, dim=1)
        s_l = float(self.exponents()[l])
        for ee in range(E):
            U = torch.rand((B, H), generator=g, device=self.device, dtype=torch.float64)
            rho = 1.0 + torch.floor(U * (Ts[:, None] + t + 1).double())
            k += (-s_l * torch.log(rho)).float()[:, :, None] * u[:, :, ee]
        return q.to(self.dtype), k.to(self.dtype), v.to(self.dtype)
