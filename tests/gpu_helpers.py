"""Helpers for the GPU parity tests: host<->device transfer of bf16 bit
patterns, and the comparison rules that allow near-tie differences."""
import numpy as np

BLK = 64


def torch():
    import torch as _t
    return _t


def dev_bf16(a: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(t.bfloat16)


def dev(a: np.ndarray):
    return torch().from_numpy(np.ascontiguousarray(a)).cuda()


def host_bits(x) -> np.ndarray:
    return x.view(torch().int16).cpu().numpy().view(np.uint16)


def host(x) -> np.ndarray:
    return x.cpu().numpy()


def meta_to_gpu(m: np.ndarray) -> np.ndarray:
    """The oracle's block metadata [.., w, d] (K-mean w = 1; Quest rows min,
    max) in the library's layout [.., d, w] (Quest: per channel the pair
    (min, max)); a relayout only, no arithmetic."""
    return np.ascontiguousarray(np.swapaxes(m, -1, -2))


def meta_from_gpu(m: np.ndarray) -> np.ndarray:
    """The library's metadata [.., d, w] in the oracle's layout [.., w, d]."""
    return np.ascontiguousarray(np.swapaxes(m, -1, -2))


def dev_meta(m: np.ndarray):
    return dev_bf16(meta_to_gpu(m))


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def attention_error(gpu_bits: np.ndarray, ref: np.ndarray):
    """max-abs and RMS error of bf16 GPU output against an fp64 reference."""
    g = bf16_to_f64(gpu_bits)
    d = g - ref
    return float(np.abs(d).max()), float(np.sqrt(np.mean(d * d)))


from oracle.compare import kept as kept_prefix, near_tie_ok  # noqa: E402,F401  (one shared rule)
