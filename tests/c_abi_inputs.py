"""The seeded inputs of the plain C driver (tests/c_abi/jorge_c_driver.c),
reproduced exactly in NumPy: u(s, t, l, i) = (int)(z >> 40) / 2^23 - 1 with
z = splitmix64(splitmix64(s * 2^32 + t * 2^16 + l) + i), splitmix64 as
published by Steele, Lea and Flood (2014). Arithmetic is on uint64 with
wrap-around, as in C."""
import numpy as np

M64 = np.uint64(0xFFFFFFFFFFFFFFFF)


def splitmix64(x):
    x = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        x = x + np.uint64(0x9E3779B97F4A7C15)
        x = (x ^ (x >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        x = (x ^ (x >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return x ^ (x >> np.uint64(31))


def uniform(seed, t, layer, count, scale=1.0):
    """float32 array of `count` values of scale * u(seed, t, layer, i)."""
    with np.errstate(over="ignore"):
        base = splitmix64(np.uint64((seed << 32) + (t << 16) + layer))
        z = splitmix64(base + np.arange(count, dtype=np.uint64))
    q = (z >> np.uint64(40)).astype(np.int32).astype(np.float32)
    return np.float32(scale) * (q / np.float32(8388608.0) - np.float32(1.0))
