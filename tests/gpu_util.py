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


def fill_pool(bd, ctx, pool, layer, lengths, ks, vs, rid_base=0, max_blocks=None,
              tables=None):
    """Give every request ceil(L/16) blocks from the pool's allocator (or use
    the given tables), write its logical K/V into those slots and return the
    block table (int32 [B, max_blocks], -1 padded)."""
    import torch
    B = len(lengths)
    need = [(int(L) + 15) // 16 for L in lengths]
    mb = max_blocks or max(1, max(need))
    if tables is None:
        tables = np.full((B, mb), -1, dtype=np.int32)
        for b in range(B):
            if need[b]:
                got = bd.boost_kv_alloc(pool, rid_base + b, need[b])
                assert got != bd.EAGAIN
                tables[b, :need[b]] = got
    slots, kk, vv = [], [], []
    for b in range(B):
        L = int(lengths[b])
        if L == 0:
            continue
        t = np.arange(L)
        slots.append(tables[b, t // 16] * 16 + t % 16)
        kk.append(ks[b])
        vv.append(vs[b])
    if slots:
        s = torch.from_numpy(np.concatenate(slots).astype(np.int32)).cuda()
        k = to_dev_u16(np.concatenate(kk))
        v = to_dev_u16(np.concatenate(vv))
        bd.boost_kv_write(ctx, pool, layer, s, k, v, int(s.numel()), stream())
        sync()
    return tables
