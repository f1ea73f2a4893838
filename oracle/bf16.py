"""bf16 bit patterns -> float64, exactly (every bf16 value is an fp64 value)."""
import numpy as np


def bf16_to_f64(bits) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 (exact widening)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)
