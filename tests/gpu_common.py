"""Helpers for the GPU parity tests: device/oracle plumbing and the tolerance checks."""
import sys

import numpy as np
import pytest
import torch


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2608_01847_amd import focus
    focus.lib()  # fails loudly if the HIP library is not built
    return focus


def announce(msg: str) -> None:
    """Names the case before a GPU step, so a fault can be attributed."""
    sys.stdout.write(f"\n[gpu-case] {msg}\n")
    sys.stdout.flush()


def host_f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float32).contiguous().numpy()


def host_bits16(t: torch.Tensor) -> np.ndarray:
    assert t.dtype == torch.bfloat16
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def host_bits32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().to(torch.float32).numpy().view(np.uint32)


def oracle_bits(values_f32: np.ndarray, dtype: torch.dtype) -> np.ndarray:
    """Bit pattern the GPU tensor must have: bf16 bits of already-bf16 values, or fp32 bits."""
    from oracle import focus_oracle as O
    if dtype == torch.bfloat16:
        return O.bf16_bits(O.bf16_round(values_f32))
    return np.ascontiguousarray(values_f32, np.float32).view(np.uint32)


def device_bits(t: torch.Tensor) -> np.ndarray:
    return host_bits16(t) if t.dtype == torch.bfloat16 else host_bits32(t)


def to_k_slabs(codes):
    """Packed codes [rows][K/2] rearranged into K-slabs [K/128][rows][64] (data movement only)."""
    rows, half = codes.shape
    assert half % 64 == 0
    if isinstance(codes, torch.Tensor):
        return codes.reshape(rows, half // 64, 64).transpose(0, 1).contiguous()
    return np.ascontiguousarray(np.asarray(codes).reshape(rows, half // 64, 64).transpose(1, 0, 2))


def assert_bits_equal(got: np.ndarray, ref: np.ndarray, what: str) -> None:
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    bad = np.nonzero(got.ravel() != ref.ravel())[0]
    assert bad.size == 0, f"{what}: {bad.size} mismatches, first at {bad[:5]}: got {got.ravel()[bad[:5]]} " \
                          f"expected {ref.ravel()[bad[:5]]}"


def rel_errors(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = max(float(np.sqrt(np.mean(ref * ref))), 1e-300)
    elem = float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), scale))) if ref.size else 0.0
    norm = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
    return elem, norm


def assert_close(got, ref, tol: float, what: str):
    """Element-wise |g - r| <= tol * max(|r|, rms(r)) and norm-wise ||g - r|| <= tol ||r||."""
    elem, norm = rel_errors(got, ref)
    assert elem <= tol and norm <= tol, f"{what}: element rel err {elem:.3e}, norm rel err {norm:.3e} > {tol}"
    return elem, norm
