"""Shared helpers of the GPU parity tests (not collected by pytest)."""
import sys

import numpy as np
import torch

import oracle

BF16_TOL_ABS = 2e-2   # max |gpu - oracle| for bf16 inputs, fp32 accumulation
F32_TOL_REL = 1e-5    # max |gpu - oracle| <= 1e-5 * max |oracle| for fp32 inputs


def device():
    assert torch.cuda.is_available(), "GPU tests need a GPU (run with -m 'not gpu' on CPU)"
    return torch.device("cuda:0")


def say(msg: str) -> None:
    """Name the case before a GPU step, so a fault can be traced to it."""
    print(msg, file=sys.stderr, flush=True)


def to_dev(a: np.ndarray) -> torch.Tensor:
    """numpy -> GPU tensor; uint16 arrays are bf16 bit patterns."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device())
    return torch.from_numpy(a).to(device())


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def bits(t: torch.Tensor) -> np.ndarray:
    """Raw bits of a GPU tensor as unsigned integers (NaN-safe comparisons)."""
    c = t.cpu().contiguous()
    if c.dtype == torch.bfloat16:
        return c.view(torch.int16).numpy().view(np.uint16)
    return c.view(torch.int32).numpy().view(np.uint32)


def attn_error(got: np.ndarray, ref: np.ndarray) -> float:
    assert got.shape == ref.shape
    assert np.isfinite(got).all()
    return float(np.max(np.abs(got - ref))) if got.size else 0.0


def assert_attn_close(out: torch.Tensor, ref: np.ndarray, what: str = "") -> float:
    got = to_f64(out)
    err = attn_error(got, ref)
    if out.dtype == torch.bfloat16:
        assert err <= BF16_TOL_ABS, f"{what}: max abs err {err} > {BF16_TOL_ABS}"
    else:
        scale = float(np.max(np.abs(ref))) if ref.size else 0.0
        assert err <= F32_TOL_REL * max(scale, 1e-30), f"{what}: max err {err} > {F32_TOL_REL}*{scale}"
    return err


def oracle_attn(d: dict) -> np.ndarray:
    return oracle.cross_attn(d["q"], d["K"], d["V"], d["src_len"])
