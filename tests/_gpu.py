"""Helpers for the GPU parity tests: move seeded inputs to the device, call the
HIP path through the C ABI binding, and bring results back as NumPy."""
import sys
import time

import numpy as np
import torch


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to("cuda").view(torch.bfloat16)


def gpu_quantize(bits, s32=None, ldx_pad=0):
    import paper_2605_31035_amd as M
    x = dev_bf16(bits)
    if ldx_pad:
        rows, k = bits.shape
        big = torch.zeros((rows, k + ldx_pad), dtype=torch.bfloat16, device="cuda")
        big[:, :k] = x
        x = big[:, :k]
    ts = None if s32 is None else torch.tensor([np.float32(s32)], dtype=torch.float32, device="cuda")
    codes, scales, s = M.mixfp4_quantize(x, ts)
    torch.cuda.synchronize()
    return codes, scales, s


def host(t):
    return t.cpu().numpy()


def dev_u8(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to("cuda")


def dev_f32(v) -> torch.Tensor:
    return torch.tensor([np.float32(v)], dtype=torch.float32, device="cuda")
