"""Small conversions shared by the tests (no method arithmetic)."""
import numpy as np
import torch


def to_bf16_bits(x) -> np.ndarray:
    """float array -> bf16 bit patterns (round to nearest even), as uint16."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def rand_bf16(rng, shape, scale=1.0, loc=0.0) -> np.ndarray:
    return to_bf16_bits(loc + scale * rng.standard_normal(shape))
