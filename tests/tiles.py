"""Small numpy tile generators for the oracle self-tests (distribution shapes of the
workloads; independent of the GPU generators)."""
import numpy as np


def tile(kind: str, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((128, 128))
    if kind == "tinyK":
        return z * np.exp(rng.standard_normal(128))[None, :] * np.exp(0.5 * rng.standard_normal(128))[:, None]
    if kind == "tinyV":
        return z * np.exp(0.5 * rng.standard_normal(128))[:, None]
    if kind == "stressK":
        t3 = z / np.sqrt((rng.standard_normal((128, 128, 3)) ** 2).sum(-1) / 3.0)
        return t3 * np.exp(1.5 * rng.standard_normal(128))[None, :]
    raise ValueError(kind)
