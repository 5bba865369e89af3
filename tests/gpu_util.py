"""Small helpers for the GPU tests (device buffers through torch)."""
import numpy as np


def to_dev_u16(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def dev_f32(*shape):
    import torch
    return torch.empty(shape, dtype=torch.float32, device="cuda")


def dev_u16(*shape):
    import torch
    return torch.empty(shape, dtype=torch.int16, device="cuda")


def host_u16(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def sync():
    import torch
    torch.cuda.synchronize()
