"""Helpers shared by the GPU parity tests: host <-> device transfers of bf16
bit arrays, and the W8A8 / protected-path tolerance checks."""
from __future__ import annotations

import numpy as np
import torch

from bf16ref import bf16_to_f64, ulp_distance

DEV = torch.device("cuda:0")


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(DEV).view(torch.bfloat16)


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy()


# Floor for cancellation: the GPU forms float(acc) * (s_tok * s_ch) + bias in
# binary32 (two roundings in the product, one in the add, one in converting an
# |acc| > 2^24), each at most 2^-24 relative to |product| or |bias|; 2^-20
# leaves a factor of four.
W8A8_CANCEL_FLOOR = 2.0 ** -20


def check_w8a8_output(y_gpu, y_ref, acc, xs, ws, bias, max_ulp=2):
    """Pass where the bf16 ulp distance is <= max_ulp or, under
    cancellation, the difference is within the binary32 floor."""
    d = ulp_distance(y_gpu, y_ref)
    prod = np.abs(acc.astype(np.float64) * xs.astype(np.float64)[:, None]
                  * ws.astype(np.float64)[None, :])
    b = 0.0 if bias is None else np.abs(bf16_to_f64(bias))[None, :]
    floor = W8A8_CANCEL_FLOOR * (prod + b)
    diff = np.abs(bf16_to_f64(y_gpu) - bf16_to_f64(y_ref))
    bad = (d > max_ulp) & (diff > floor)
    assert not bad.any(), (
        f"{int(bad.sum())} outputs beyond tolerance; max ulp {int(d.max())}, "
        f"first at {np.argwhere(bad)[0].tolist()}")
    return int(d.max()), float((d == 0).mean())


def check_bf16_output(y_gpu, X, W, bias, rel_frob=2.0 ** -8):
    """Protected path against binary64 X W^T + b: elementwise within one bf16
    ulp plus the binary32 summation bound K 2^-23 sum|x w|, and overall
    within rel_frob (bf16 output rounding alone is ~2^-10 rms)."""
    Xf = bf16_to_f64(X).reshape(X.shape)
    Wf = bf16_to_f64(W).reshape(W.shape)
    K = Xf.shape[1]
    ref = Xf @ Wf.T
    if bias is not None:
        ref = ref + bf16_to_f64(bias)[None, :]
    mag = np.abs(Xf) @ np.abs(Wf).T
    y = bf16_to_f64(y_gpu).reshape(ref.shape)
    ulp = np.maximum(np.abs(ref), 2.0 ** -126) * 2.0 ** -7
    bound = ulp + K * 2.0 ** -23 * mag
    assert np.all(np.abs(y - ref) <= bound)
    rel = np.linalg.norm(y - ref) / np.linalg.norm(ref)
    assert rel <= rel_frob, rel
    return rel
