"""Small random models and contexts for the oracle's CPU pins (fp64 NumPy)."""
import numpy as np

import oracle


def small_model(seed=0, L=2, D=32, hq=4, hkv=2, hd=8, F=48, V=64, theta=10000.0, std=0.3,
                random_gains=True):
    """Weights in the library layout, as fp64 arrays. Norm gains are random unless asked."""
    rng = np.random.default_rng(seed)
    dims = oracle.ModelDims(L, D, hq, hkv, hd, F, theta, 1e-6)
    g = (lambda n: 1.0 + 0.3 * rng.standard_normal(n)) if random_gains else (lambda n: np.ones(n))
    layers = []
    for _ in range(L):
        layers.append({
            "attn_norm": g(D),
            "w_qkv": std * rng.standard_normal(((hq + 2 * hkv) * hd, D)),
            "w_o": std * rng.standard_normal((D, hq * hd)),
            "mlp_norm": g(D),
            "w_gate_up": std * rng.standard_normal((2 * F, D)),
            "w_down": std * rng.standard_normal((D, F)),
        })
    weights = {"embed": rng.standard_normal((V, D)), "final_norm": g(D), "layers": layers}
    return dims, weights, V


def context(seed, lens, q, V):
    rng = np.random.default_rng(seed + 7)
    return rng.integers(0, V, size=int(sum(lens)) + q)
