"""Seeded int4 layer weights drawn on the GPU with torch, for runs that only
time or self-check the path (the 80-layer step, whose 35 GB of weights would
take minutes to draw on the host).  Same recipe as gen.w4_random: W ~ N(0,
std) rounded to fp16, then per-(row, 128-group) asymmetric min/max
quantisation s = fp16((max - min) / 15) (1 if 0), z = clamp(rne(-min / s), 0,
15), q = clamp(rne(w / s) + z, 0, 15), nibbles packed low = even k.  The
random stream is torch's, not gen's, so these weights are never compared
against the reference."""
from __future__ import annotations


def w4_random_device(seed: int, stream: int, N: int, K: int, std: float = 0.02, device="cuda"):
    """(qweight u8 [N][K/2], scales fp16 bits int16 [N][K/128], zeros u8 [N][K/128]) on `device`."""
    import torch
    assert K % 128 == 0
    g = torch.Generator(device=device)
    g.manual_seed((seed << 20) + stream)
    q = torch.empty((N, K // 2), dtype=torch.uint8, device=device)
    s_out = torch.empty((N, K // 128), dtype=torch.float16, device=device)
    z_out = torch.empty((N, K // 128), dtype=torch.uint8, device=device)
    rows = max(1, (1 << 26) // K)  # bound the fp32 temporaries
    for r0 in range(0, N, rows):
        n = min(rows, N - r0)
        w = (torch.randn((n, K), generator=g, device=device, dtype=torch.float32) * std).half().float()
        wg = w.view(n, K // 128, 128)
        mn, mx = wg.amin(-1), wg.amax(-1)
        s = ((mx - mn) / 15).half()
        s = torch.where(s == 0, torch.ones_like(s), s)
        sf = s.float()
        z = torch.clamp(torch.round(-mn / sf), 0, 15)
        qq = torch.clamp(torch.round(wg / sf[..., None]) + z[..., None], 0, 15).to(torch.uint8).view(n, K)
        q[r0:r0 + n] = qq[:, 0::2] | (qq[:, 1::2] << 4)
        s_out[r0:r0 + n] = s
        z_out[r0:r0 + n] = z.to(torch.uint8)
    return q, s_out.view(torch.int16), z_out


def normal_f16_device(seed: int, stream: int, shape, mean: float = 0.0, std: float = 1.0, device="cuda"):
    """fp16 N(mean, std) draws as int16 bits on `device` (torch's stream)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed << 20) + stream)
    return (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std + mean).half().view(torch.int16)
