"""Seeded numpy tile generators (input shapes only, none of the method's arithmetic): the
workload distributions for the oracle self-tests, and the structured tiles of the property
tests, which feed both the oracle and the GPU path."""
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


STRUCTURES = ("gauss", "outlier_channels", "outlier_tokens", "constant_rows", "constant_cols", "zeros",
              "single_outlier", "heavy_tail", "sparse")


def make_tile(structure: str, seed: int, log_scale: float) -> np.ndarray:
    """One 128-token x 128-channel tile (token-major) of the given structure, times 10^log_scale."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((128, 128))
    if structure == "gauss":
        X = z
    elif structure == "outlier_channels":
        X = z * np.exp(1.5 * rng.standard_normal(128))[None, :]
    elif structure == "outlier_tokens":
        X = z * np.exp(1.5 * rng.standard_normal(128))[:, None]
    elif structure == "constant_rows":
        X = np.repeat(rng.standard_normal((128, 1)), 128, axis=1)
    elif structure == "constant_cols":
        X = np.repeat(rng.standard_normal((1, 128)), 128, axis=0)
    elif structure == "zeros":
        X = np.zeros((128, 128))
    elif structure == "single_outlier":
        X = np.zeros((128, 128))
        X[rng.integers(128), rng.integers(128)] = 40.0 * rng.choice([-1.0, 1.0])
    elif structure == "heavy_tail":
        X = rng.standard_t(2.0, (128, 128))
    else:  # sparse
        X = z * (rng.random((128, 128)) < 0.05)
    return X * 10.0 ** log_scale
