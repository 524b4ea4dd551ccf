"""Seeded synthetic decode workloads for the ReTopK selector.

This module only draws random numbers and rounds them to the storage dtype.  It
holds none of the method's arithmetic, so both the GPU path and the CPU oracle
can consume its arrays.

Keys of KV head g are clustered: ``k_i = 2 c_{g, z_i} + N(0, I)`` with centres
``c ~ N(0, I/d)`` and ``z_i`` uniform over the head's centres; values are
``N(0, I)``.  Each query head follows a walk on the sphere of radius sqrt(d):
``q_0 = sqrt(d) * c_hat_{g, z_0}``, then either (probability p_jump) a jump
``q_u = sqrt(d) * c_hat_{g, z}`` to a uniformly drawn centre, or an AR(1) move
``q_u = sqrt(d) * unit(alpha q_{u-1} + 0.436 xi)``, ``xi ~ N(0, I)``.  The first
``cache_cap`` walk entries are the prompt-tail queries at positions
``prompt_len - cache_cap .. prompt_len - 1``; the next ``steps`` entries are the
decode queries.  The paper measures on real model activations (PG19 and RULER
contexts on Qwen2.5 / Llama-3.1); these inputs stand in for them.

bf16 workloads are rounded once (round to nearest even) on the host; the same
bits feed the GPU and, widened exactly to float32, the oracle.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str          # "f32" or "bf16"
    prompt_len: int     # N: KV rows present before the first decode step
    steps: int          # T: decode steps (one KV row appended per step)
    k: int              # K: support size
    cache_cap: int      # C (paper) / M: query-support cache capacity
    r: int              # R (paper): retrieved cache entries per step
    window: int         # W: recent window
    tau: float          # similarity fallback threshold
    refresh: int        # T_r (paper) / P: refresh period, 0 = off
    n_centers: int      # key clusters per KV head
    alpha: float        # AR(1) coefficient of the query walk
    p_jump: float       # probability of a jump to a random centre
    seed: int = 0

    @property
    def max_len(self) -> int:
        return self.prompt_len + self.steps

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def step_len(self, t: int) -> int:
        """KV length seen by decode step t: the prompt plus t+1 appended rows."""
        return self.prompt_len + t + 1

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    # fp32, one head: the size the oracle finishes in seconds.
    "tiny": Workload("tiny", 1, 1, 1, 64, "f32", 2048, 64, 32, 64, 4, 64, 0.8, 16, 16, 0.9, 0.1),
    # One attention layer, 32 query heads on 8 KV heads, bf16.
    "16k": Workload("16k", 1, 32, 8, 128, "bf16", 16384, 128, 256, 256, 4, 128, 0.8, 32, 64,
                    0.9, 0.05),
    "32k": Workload("32k", 1, 32, 8, 128, "bf16", 32768, 256, 512, 256, 8, 128, 0.8, 32, 128,
                    0.9, 0.05),
    # The headline layer: 128K context, K=512.
    "128k": Workload("128k", 1, 32, 8, 128, "bf16", 131072, 256, 512, 512, 8, 256, 0.8, 64, 256,
                     0.9, 0.05),
    # The headline layer with the paper's default selector settings (Sec. 4.1:
    # C = W = 32, R = 4, tau = 0.85, T_r = 128).
    "128k_paper": Workload("128k_paper", 1, 32, 8, 128, "bf16", 131072, 256, 512, 32, 4, 32,
                           0.85, 128, 256, 0.9, 0.05),
    # The layer layout of the paper's main model (Qwen2.5-7B: 28 query heads on 4
    # KV heads, d = 128) at 128K with the default selector settings.
    "128k_28x4_paper": Workload("128k_28x4_paper", 1, 28, 4, 128, "bf16", 131072, 256, 512, 32,
                                4, 32, 0.85, 128, 256, 0.9, 0.05),
    # Fallback-heavy: four sequences at 64K, frequent jumps, tau = 0.9.
    "stress": Workload("stress", 4, 32, 8, 128, "bf16", 65536, 256, 1024, 512, 8, 256, 0.9, 16,
                       256, 0.9, 0.3),
}


# ---------------------------------------------------------------------------
# bf16 storage
# ---------------------------------------------------------------------------

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even. Finite inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(
        np.float32)


@dataclass
class Inputs:
    """All arrays of one workload.

    ``*_f32`` arrays hold the exact values (float32) that both sides use; for
    bf16 workloads ``*_raw`` holds the uint16 bit patterns the GPU consumes,
    for f32 workloads ``*_raw`` is the float32 array itself.
    """
    w: Workload
    q_tail_raw: np.ndarray   # [B, Hq, C, d]
    q_dec_raw: np.ndarray    # [T, B, Hq, d]
    k_raw: np.ndarray        # [B, Hkv, max_len, d]
    v_raw: np.ndarray        # [B, Hkv, max_len, d]
    centre_of_key: np.ndarray    # [B, Hkv, max_len] int32 cluster label z_i
    centre_of_query: np.ndarray  # [B, Hq, C + T] int32 last centre the walk jumped to

    def f32(self, name: str) -> np.ndarray:
        a = getattr(self, name + "_raw")
        return bf16_bits_to_f32(a) if a.dtype == np.uint16 else a

    @property
    def q_tail(self) -> np.ndarray:
        return self.f32("q_tail")

    @property
    def q_dec(self) -> np.ndarray:
        return self.f32("q_dec")

    @property
    def k(self) -> np.ndarray:
        return self.f32("k")

    @property
    def v(self) -> np.ndarray:
        return self.f32("v")


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def make_inputs(w: Workload, seed: int | None = None) -> Inputs:
    """Draw every array of workload `w` from one seed (default: the workload's)."""
    seed = w.seed if seed is None else seed
    ss = np.random.SeedSequence(seed)
    s_centre, s_assign, s_knoise, s_val, s_query = ss.spawn(5)
    g_centre = np.random.Generator(np.random.PCG64(s_centre))
    g_assign = np.random.Generator(np.random.PCG64(s_assign))
    g_knoise = np.random.Generator(np.random.PCG64(s_knoise))
    g_val = np.random.Generator(np.random.PCG64(s_val))
    g_query = np.random.Generator(np.random.PCG64(s_query))

    B, Hq, Hkv, d, L = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_len
    sdt = np.uint16 if w.dtype == "bf16" else np.float32
    k_raw = np.empty((B, Hkv, L, d), sdt)
    v_raw = np.empty((B, Hkv, L, d), sdt)
    z_all = np.empty((B, Hkv, L), np.int32)
    centres = np.empty((B, Hkv, w.n_centers, d), np.float64)

    for b in range(B):
        for g in range(Hkv):
            c = g_centre.standard_normal((w.n_centers, d)) / np.sqrt(d)
            centres[b, g] = c
            z = g_assign.integers(0, w.n_centers, size=L, dtype=np.int64)
            z_all[b, g] = z
            keys = (2.0 * c[z]).astype(np.float32)
            keys += g_knoise.standard_normal((L, d), dtype=np.float32)
            k_raw[b, g] = _store(keys, w.dtype)
            del keys
            vals = g_val.standard_normal((L, d), dtype=np.float32)
            v_raw[b, g] = _store(vals, w.dtype)
            del vals

    n_walk = w.cache_cap + w.steps
    walk = np.empty((B, Hq, n_walk, d), np.float32)
    walk_centre = np.empty((B, Hq, n_walk), np.int32)
    sqrt_d = np.sqrt(d)
    noise_scale = 0.436
    for b in range(B):
        for h in range(Hq):
            g = h // w.group
            chat = centres[b, g] / np.linalg.norm(centres[b, g], axis=1, keepdims=True)
            z = int(g_query.integers(0, w.n_centers))
            q = sqrt_d * chat[z]
            for u in range(n_walk):
                if u > 0:
                    if g_query.random() < w.p_jump:
                        z = int(g_query.integers(0, w.n_centers))
                        q = sqrt_d * chat[z]
                    else:
                        x = w.alpha * q + noise_scale * g_query.standard_normal(d)
                        q = sqrt_d * x / np.linalg.norm(x)
                walk[b, h, u] = q
                walk_centre[b, h, u] = z

    q_tail = walk[:, :, :w.cache_cap]                     # [B, Hq, C, d]
    q_dec = np.transpose(walk[:, :, w.cache_cap:], (2, 0, 1, 3))   # [T, B, Hq, d]
    return Inputs(
        w=w,
        q_tail_raw=_store(np.ascontiguousarray(q_tail), w.dtype),
        q_dec_raw=_store(np.ascontiguousarray(q_dec), w.dtype),
        k_raw=k_raw,
        v_raw=v_raw,
        centre_of_key=z_all,
        centre_of_query=walk_centre,
    )


def make_support_state(inp: Inputs, seed: int = 1,
                       heads: list[int] | None = None) -> tuple[np.ndarray, np.ndarray]:
    """A seeded, valid cache of supports without running any selection.

    For each (sequence, query head) and cache slot u (holding prompt-tail query u),
    draws K distinct key indices below the query's causal length, half of them from
    the key cluster the query walked to and the rest uniformly.  Returns
    (supp [B*Hq, C, K] int32 ascending, cnt [B*Hq, C] int32).  It lets a full-size
    test start a decode step from a plausible cache state at once.  With `heads`
    (flat b*Hq + h indices) only those heads are drawn; the others hold empty
    supports.
    """
    w = inp.w
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    C, K = w.cache_cap, w.k
    supp = np.full((w.batch * w.n_q_heads, C, K), -1, np.int32)
    cnt = np.zeros((w.batch * w.n_q_heads, C), np.int32)
    for b in range(w.batch):
        for h in range(w.n_q_heads):
            if heads is not None and b * w.n_q_heads + h not in heads:
                continue
            g = h // w.group
            cnt[b * w.n_q_heads + h] = K
            zk = inp.centre_of_key[b, g]
            for u in range(C):
                lim = w.prompt_len - C + u + 1
                members = np.flatnonzero(zk[:lim] == inp.centre_of_query[b, h, u])
                take = rng.permutation(members)[:K // 2]
                chosen = set(int(i) for i in take)
                while len(chosen) < K:
                    chosen.update(int(i) for i in rng.integers(0, lim, size=K - len(chosen)))
                supp[b * w.n_q_heads + h, u] = np.sort(np.fromiter(chosen, np.int32, K))
    return supp, cnt
