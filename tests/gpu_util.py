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


def slices_sum(flat, S, B, N, K):
    """The output [B, N] that a split-K slice buffer stands for, by the layout
    and order the library's header states: S slices [S][B][N] added in slice
    order to 0.0f (fp32 adds), and for a row of the [N, K] matrix that
    crosses a 2 MiB page, the sum of its earlier page's parts plus the sum of
    its later page's parts, kept after the slices by the page of the row's
    last column.  One slice is the output itself."""
    flat = np.asarray(flat, np.float32)
    if S == 1:
        return flat[:B * N].reshape(B, N).copy()
    sl = flat[:S * B * N].reshape(S, B, N)
    acc = np.zeros((B, N), np.float32)
    for s in range(S):
        acc = acc + sl[s]
    tail = flat[S * B * N:]
    page = 1 << 20
    for r in range(N):
        first, last = r * K // page, (r * K + K - 1) // page
        if first == last:
            continue
        v0, v1 = np.zeros(B, np.float32), np.zeros(B, np.float32)
        for s in range(S):
            o0, o1 = ((last * 2) * S + s) * B, ((last * 2 + 1) * S + s) * B
            v0 = v0 + tail[o0:o0 + B]
            v1 = v1 + tail[o1:o1 + B]
        acc[:, r] = v0 + v1
    return acc
