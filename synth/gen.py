"""Seeded synthetic Q/K/V generator shared by the oracle tests, the GPU tests
and the benchmark.

It holds none of the method's arithmetic: it only draws inputs.

Each channel of each head is a smooth space-time field plus noise, the way
video-DiT activations vary slowly across neighbouring latent tokens:

    X[t, y, x, c] = s_X,h * sum_{k<4} a_k sin(2 pi (kt t/T + ky y/Hg + kx x/Wg) + phi_k(t))
                    + 0.1 * eps

with integer wave numbers kt in {0,1,2}, ky, kx in {0..3}, a_k ~ N(0,1),
phi_k ~ U[0, 2 pi), eps ~ N(0,1). Q and K share their wave vectors per
(head, channel, k) with independent amplitudes and phases, so logits depend
on the displacement between tokens; V is independent. Optional features:
per-head scale s ~ U[0.5, 2]; 1% key outliers scaled by 8; phases drifting
linearly over frames (phi_k(t) = phi_k + omega_k t, omega_k ~ U[-pi/8, pi/8]).

Token order is frame-major raster: n = t*Hg*Wg + y*Wg + x. Tensors are
returned as float32 numpy arrays of shape [B, H, N, d]; for bf16 workloads
the values are already rounded to bf16 (round to nearest even), so the
float32 array holds exactly the values the GPU sees.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

N_WAVES = 4
NOISE_STD = 0.1


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); return float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def _field(rng, waves, T, Hg, Wg, d, scale, drift):
    """One head of one tensor: [N, d] float32.

    Each wave is separable over (t, y, x): sin(theta) is the imaginary part of
    exp(i(phi + omega t + 2 pi kt t/T)) exp(i 2 pi ky y/Hg) exp(i 2 pi kx x/Wg),
    so the field is one complex contraction over the waves instead of one sine
    per token, channel and wave."""
    kt, ky, kx = waves                                   # each [d, 4] ints
    amp = rng.standard_normal((d, N_WAVES))
    phi = rng.uniform(0.0, 2 * np.pi, (d, N_WAVES))
    omega = rng.uniform(-np.pi / 8, np.pi / 8, (d, N_WAVES)) if drift else np.zeros((d, N_WAVES))
    noise = rng.standard_normal((T * Hg * Wg, d)).astype(np.float32)
    t = np.arange(T, dtype=np.float64)[:, None, None]
    y = np.arange(Hg, dtype=np.float64)[:, None, None]
    x = np.arange(Wg, dtype=np.float64)[:, None, None]
    ft = amp * np.exp(1j * (phi + (omega + 2 * np.pi * kt / T) * t))     # [T, d, 4]
    fy = np.exp(1j * (2 * np.pi * ky / Hg) * y)                             # [Hg, d, 4]
    fx = np.exp(1j * (2 * np.pi * kx / Wg) * x)                             # [Wg, d, 4]
    ty = (ft[:, None] * fy[None]).reshape(T * Hg, d, N_WAVES).transpose(1, 0, 2)   # [d, T*Hg, 4]
    acc = np.matmul(ty, fx.transpose(1, 2, 0)).imag                                 # [d, T*Hg, Wg]
    out = (scale * acc).reshape(d, T * Hg * Wg).T.astype(np.float32)
    out += np.float32(NOISE_STD) * noise
    return out


def generate(w, heads=None):
    """Draw Q, K, V for workload ``w`` (a ``synth.configs.Workload``).

    ``heads`` optionally restricts generation to a subset of head indices
    (the draws for a head do not depend on which other heads are drawn).
    Returns float32 arrays [B, len(heads), N, d].
    """
    heads = list(range(w.H)) if heads is None else list(heads)
    T, Hg, Wg, d, N = w.T, w.Hg, w.Wg, w.d, w.N
    shape = (w.B, len(heads), N, d)
    Q = np.empty(shape, np.float32)
    K = np.empty(shape, np.float32)
    V = np.empty(shape, np.float32)

    def one(b, hi, h):
        ss = np.random.SeedSequence([w.seed, b, h])
        r_w, r_s, r_q, r_k, r_v, r_o = [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(6)]
        waves_qk = (r_w.integers(0, 3, (d, N_WAVES)), r_w.integers(0, 4, (d, N_WAVES)),
                    r_w.integers(0, 4, (d, N_WAVES)))
        waves_v = (r_w.integers(0, 3, (d, N_WAVES)), r_w.integers(0, 4, (d, N_WAVES)),
                   r_w.integers(0, 4, (d, N_WAVES)))
        if w.head_scale:
            sq, sk, sv = r_s.uniform(0.5, 2.0, 3)
        else:
            sq = sk = sv = 1.0
        Q[b, hi] = _field(r_q, waves_qk, T, Hg, Wg, d, sq, w.phase_drift)
        K[b, hi] = _field(r_k, waves_qk, T, Hg, Wg, d, sk, w.phase_drift)
        V[b, hi] = _field(r_v, waves_v, T, Hg, Wg, d, sv, w.phase_drift)
        if w.key_outliers > 0:
            n_out = int(round(w.key_outliers * N))
            idx = r_o.choice(N, size=n_out, replace=False)
            K[b, hi, idx] *= np.float32(8.0)
        if w.dtype == "bf16":
            for X in (Q, K, V):
                X[b, hi] = round_to_bf16(X[b, hi])

    # every head draws from its own seed, so the heads can be drawn in parallel
    jobs = [(b, hi, h) for b in range(w.B) for hi, h in enumerate(heads)]
    workers = min(len(jobs), 8, os.cpu_count() or 1)
    if workers > 1:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(lambda j: one(*j), jobs))
    else:
        for j in jobs:
            one(*j)
    return Q, K, V
