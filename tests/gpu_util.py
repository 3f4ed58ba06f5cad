"""Helpers for the GPU parity tests: device buffers with poisoned guard bands,
bit-pattern transfers, and seeded device-side input generation.

Inputs generated here come from torch's seeded generators (input generation
only); the oracle always receives a host copy of the same bits.  Nothing in
this module computes any result of the method.
"""

from __future__ import annotations

import numpy as np
import torch

GUARD_BYTES = 4096
POISON16 = 0xFFFF            # a NaN pattern no kernel writes for data or padding
DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


def step(msg: str) -> None:
    """Name the case before a GPU step, so a crash log says where it was."""
    print(f"[gpu] {msg}", flush=True)


def to_dev_u16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).to(DEV).view(torch.bfloat16)


def to_dev_f32(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def host_u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1)


def host_u32(t: torch.Tensor) -> np.ndarray:
    return t.detach().view(torch.int32).cpu().numpy().view(np.uint32).reshape(-1)


class Guarded:
    """A device buffer of ``numel`` elements inside poisoned guard bands.

    ``shift`` moves the start by that many elements (to test element-aligned,
    not 16-byte-aligned, pointers).
    """

    def __init__(self, numel: int, dtype: torch.dtype, shift: int = 0):
        esz = torch.empty(0, dtype=dtype).element_size()
        self.g = GUARD_BYTES // esz
        self.numel = numel
        self.shift = shift
        total = self.g + shift + numel + self.g
        self.raw = torch.empty(total, dtype=dtype, device=DEV)
        self.raw.view(torch.uint8).fill_(0xFF)
        self.view = self.raw[self.g + shift:self.g + shift + numel]

    def guards_intact(self) -> bool:
        b = self.raw.view(torch.uint8)
        esz = self.raw.element_size()
        lo = (self.g + self.shift) * esz
        hi = (self.g + self.shift + self.numel) * esz
        return bool((b[:lo] == 0xFF).all().item()) and bool((b[hi:] == 0xFF).all().item())


def gen(seed: int) -> torch.Generator:
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return g


def dev_random_bits16(n: int, seed: int, chunk: int = 1 << 28) -> torch.Tensor:
    """n uniformly random 16-bit words on the device (as a bf16 tensor)."""
    out = torch.empty(n, dtype=torch.int16, device=DEV)
    g = gen(seed)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        out[s:e] = torch.randint(-32768, 32768, (e - s,), dtype=torch.int16, device=DEV, generator=g)
    return out.view(torch.bfloat16)


def dev_random_f32_bits(n: int, seed: int) -> torch.Tensor:
    """n uniformly random 32-bit words on the device, as fp32 (NaNs included)."""
    g = gen(seed)
    return torch.randint(-(1 << 31), 1 << 31, (n,), dtype=torch.int64, device=DEV, generator=g) \
        .to(torch.int32).view(torch.float32)


def dev_wide_bf16(n: int, seed: int, chunk: int = 1 << 27) -> torch.Tensor:
    """n finite bf16 values with exponents spread over 2^-15..2^15 (sums round)."""
    out = torch.empty(n, dtype=torch.int16, device=DEV)
    g = gen(seed)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        m = e - s
        sign = torch.randint(0, 2, (m,), dtype=torch.int32, device=DEV, generator=g)
        expo = torch.randint(112, 143, (m,), dtype=torch.int32, device=DEV, generator=g)
        mant = torch.randint(0, 128, (m,), dtype=torch.int32, device=DEV, generator=g)
        bits = (sign << 15) | (expo << 7) | mant
        bits = torch.where(bits >= 32768, bits - 65536, bits)
        out[s:e] = bits.to(torch.int16)
    return out.view(torch.bfloat16)


def dev_wide_f32(n: int, seed: int, chunk: int = 1 << 27) -> torch.Tensor:
    """n fp32 values N(0,1) * 2^k with k uniform in [-30, 30] (sums round)."""
    out = torch.empty(n, dtype=torch.float32, device=DEV)
    g = gen(seed)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        m = e - s
        k = torch.randint(-30, 31, (m,), dtype=torch.int32, device=DEV, generator=g).to(torch.float32)
        out[s:e] = torch.randn(m, device=DEV, generator=g) * torch.exp2(k)
    return out
