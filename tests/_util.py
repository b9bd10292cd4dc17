"""Marshalling between the synthetic torch layers and the oracle's numpy arrays."""
import numpy as np
import torch


def to_np_bits(t: torch.Tensor) -> np.ndarray:
    """Tensor -> numpy; bfloat16 becomes its uint16 bit pattern, fp8 codes stay uint8."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def oracle_inputs(layer):
    """(desc, banks, logits, slot_table, x) in the form the oracle takes."""
    banks = {"w13": to_np_bits(layer.w13), "w2": to_np_bits(layer.w2)}
    if layer.s13 is not None:
        banks["s13"] = to_np_bits(layer.s13)
        banks["s2"] = to_np_bits(layer.s2)
    return (layer.desc(), banks, to_np_bits(layer.logits), to_np_bits(layer.slot_table),
            to_np_bits(layer.x))


def decode_bank_torch(bank: torch.Tensor, w_dtype: int, scales=None) -> torch.Tensor:
    """Independent (torch-based) weight decode used to cross-check the oracle."""
    if w_dtype == 0:
        return bank.double()
    if w_dtype == 1:
        return bank.to(torch.float64)
    if w_dtype == 3:
        # MXFP4: split the nibbles, decode E2M1 arithmetically (sign, 2-bit exponent with bias
        # 1, 1-bit mantissa; exponent 0 subnormal) and E8M0 through torch's own dtype
        b = bank.to(torch.int64)
        codes = torch.stack([b & 0xF, b >> 4], dim=-1).reshape(b.shape[0], -1)
        sign = torch.where(codes >= 8, -1.0, 1.0).double()
        e, m = (codes >> 1) & 3, (codes & 1).double()
        mag = torch.where(e == 0, m * 0.5, (1.0 + m * 0.5) * torch.pow(2.0, (e - 1).double()))
        s = scales.t().contiguous().view(torch.float8_e8m0fnu).to(torch.float64).repeat_interleave(32, 1)
        return sign * mag * s
    v = bank.view(torch.float8_e4m3fn).to(torch.float64)
    s = scales.double().repeat_interleave(128, 0).repeat_interleave(128, 1)
    return v * s
