"""Helpers shared by the GPU tests: moving synth's bf16 bit arrays to and from
the device, the parity gate, and case banners printed before each GPU step."""
import sys

import numpy as np

import oracle

REL_L2_MAX = 1e-3          # relative L2 error bound
MAX_ABS_FRAC = 5e-3        # max abs error bound, as a fraction of max|y_ref|


def banner(msg: str):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def dev_bf16(bits: np.ndarray):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    return t.view(torch.bfloat16).cuda()


def dev_u8(b: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(b, dtype=np.uint8)).cuda()


def host_bits(t) -> np.ndarray:
    """Device bf16/int16/uint8 tensor -> numpy array of its raw bits."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def host_f32(t) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def parity(y: np.ndarray, y_ref: np.ndarray, what: str = "", slack=None):
    """Relative L2 <= 1e-3 and |y - y_ref| <= 5e-3 * max |y_ref| per element,
    plus slack (per element) when given."""
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    assert y.shape == y_ref.shape
    assert np.all(np.isfinite(y)), what
    diff = y - y_ref
    ref_norm = np.linalg.norm(y_ref)
    rel = np.linalg.norm(diff) / ref_norm if ref_norm > 0 else np.linalg.norm(diff)
    max_ref = np.abs(y_ref).max()
    max_abs = np.abs(diff).max()
    assert rel <= REL_L2_MAX, f"{what}: relative L2 {rel:.3e} > {REL_L2_MAX}"
    bound = MAX_ABS_FRAC * max_ref + (0.0 if slack is None else slack)
    over = np.abs(diff) > bound
    assert not over.any(), (f"{what}: |y - y_ref| {np.abs(diff)[over].max():.3e} over the bound "
                            f"{MAX_ABS_FRAC} * {max_ref:.3e}" + ("" if slack is None else " + slack"))
    return rel, max_abs / max_ref if max_ref > 0 else 0.0


def bf16_ulp(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """One bf16 unit in the last place (8 significant bits) at the larger
    magnitude of a and b, element by element; 0 where both are 0."""
    m = np.maximum(np.abs(np.asarray(a, dtype=np.float64)), np.abs(np.asarray(b, dtype=np.float64)))
    e = np.floor(np.log2(np.where(m > 0, m, 1.0)))
    return np.where(m > 0, np.exp2(e - 7), 0.0)


def parity_bf16_out(y_bits: np.ndarray, y_ref: np.ndarray, what: str = ""):
    """bf16 output against the round-to-nearest-even bf16 of the fp64 result:
    the same relative L2 bound, and per element the max-abs bound plus one
    bf16 ulp -- an fp32 sum within the fp32 gate that lies near a rounding
    boundary rounds to the neighbouring bf16 value, one ulp (2^-8 to 2^-7 of
    the value, more than 5e-3 of it) from RNE_bf16(y_ref)."""
    from paper_2607_04031_amd import synth
    ref_bits = oracle.round_bf16(y_ref)
    y = synth.bf16_bits_to_f32(y_bits)
    ref = synth.bf16_bits_to_f32(ref_bits)
    return parity(y, ref, what, slack=bf16_ulp(y, ref))
