"""Calibration of the learnable rotation (Sec. 4.1.4): offline, PyTorch.

The rotation R = diag(R_1 .. R_{D/2}) of the interleaved (Sec. 4.1.2) or half
(Sec. 4.1.3) scheme is fitted to calibration Q and K by minimising

    || Y - Q4(Q_s R) Q4(K_s R)^T ||_F^2 ,   Y = Q_s K_s^T ,

where Q_s, K_s are the 3D-RoPE'd and smoothed (mean-subtracted) matrices and
Q4 the symmetric INT4 fake quantiser of the kernels (per group of tokens:
s = amax/7, code = clamp(round(x * 7/amax), -7, 7), half-to-even).  Every
block stays in O(2) by construction, as the paper requires: a block is the
reflection [[cos a, sin a], [sin a, -cos a]] (the family of H_2, which is the
angle pi/4 and the default initialisation) or the rotation
[[cos a, sin a], [-sin a, cos a]], and only its angle a is learned.  The
rounding passes gradients straight through; the group maxima pass theirs.

The result is a float64 array [D/2][2][2] to hand to the library as
``rot_blocks`` (``rotate_attn.make_params(..., rot_blocks=...)``).  The paper
reports this calibration as preliminary (with one or two samples it did not
beat the fixed half rotation); this module reproduces the procedure on
whatever data it is given, it carries no claim about accuracy.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

D = 128


def _torch():
    import torch
    return torch


def _as_float(x, device):
    """bf16 bit patterns (uint16 numpy) or a float tensor/array -> float32 tensor [..., N, D]."""
    torch = _torch()
    if isinstance(x, np.ndarray) and x.dtype == np.uint16:
        f = (x.astype(np.uint32) << 16).view(np.float32)
        return torch.from_numpy(np.ascontiguousarray(f)).to(device)
    if isinstance(x, np.ndarray):
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)
    return x.to(device=device, dtype=torch.float32)


def rope_tables(grid, split, theta, device):
    """cos/sin of every (token, pair) for the 3D RoPE of Sec. 3: token
    n = (t*Hg + h)*W + w; pair k of axis a turns by pos_a * theta^(-2k/D_a)."""
    torch = _torch()
    T, Hg, W = grid
    n = torch.arange(T * Hg * W, dtype=torch.float64)
    pos = [torch.div(n, Hg * W, rounding_mode="floor"), torch.remainder(torch.div(n, W, rounding_mode="floor"), Hg),
           torch.remainder(n, W)]
    ang = []
    for a, Da in enumerate(split):
        k = torch.arange(Da // 2, dtype=torch.float64)
        omega = float(theta) ** (-(2.0 * k) / Da)
        ang.append(pos[a][:, None] * omega[None, :])
    phi = torch.cat(ang, 1)
    return torch.cos(phi).float().to(device), torch.sin(phi).float().to(device)


def apply_rope(x, cos, sin):
    """Row-vector convention [y0 y1] = [x0 x1] [[cos, sin], [-sin, cos]] on pairs (2p, 2p+1)."""
    x0, x1 = x[..., 0::2], x[..., 1::2]
    y0 = x0 * cos - x1 * sin
    y1 = x0 * sin + x1 * cos
    return _torch().stack((y0, y1), -1).flatten(-2)


def half_permutation(split):
    """Channel order Pi of the half rotation (Sec. 4.1.3): in each segment channel
    o+i and o+i+D_a/2 become the adjacent positions (o+2i, o+2i+1)."""
    idx = []
    o = 0
    for Da in split:
        h = Da // 2
        for i in range(h):
            idx += [o + i, o + i + h]
        o += Da
    return idx


def blocks_from_angles(angles, kinds):
    """O(2) blocks [P][2][2]: kind 1 = reflection [[c, s], [s, -c]], 0 = rotation [[c, s], [-s, c]]."""
    torch = _torch()
    c, s = torch.cos(angles), torch.sin(angles)
    sigma = torch.where(kinds > 0, torch.ones_like(c), -torch.ones_like(c))
    row0 = torch.stack((c, s), -1)
    row1 = torch.stack((sigma * s, -sigma * c), -1)   # reflection [s, -c], rotation [-s, c]
    return torch.stack((row0, row1), -2)


def apply_blocks(y, R):
    """[z_2p z_2p+1] = [y_2p y_2p+1] R_p for every pair p (row-vector form)."""
    shp = y.shape
    pairs = y.reshape(*shp[:-1], shp[-1] // 2, 1, 2)
    return (pairs @ R).reshape(shp)


def fake_quant(x, group):
    """Symmetric INT4 per group of `group` consecutive tokens (rows of the last two
    dims), straight-through rounding: s = amax/7, clamp(round(x * 7/amax), -7, 7) * s."""
    torch = _torch()
    N = x.shape[-2]
    pad = (-N) % group
    xp = torch.nn.functional.pad(x, (0, 0, 0, pad)) if pad else x
    g = xp.reshape(*xp.shape[:-2], (N + pad) // group, group * xp.shape[-1])
    amax = g.abs().amax(-1, keepdim=True)
    safe = torch.where(amax > 0, amax, torch.ones_like(amax))
    inv = 7.0 / safe
    t = g * inv
    r = t + (torch.round(t) - t).detach()
    q = torch.clamp(r, -7.0, 7.0) * (safe / 7.0)
    q = torch.where(amax > 0, q, torch.zeros_like(q))
    return q.reshape(xp.shape)[..., :N, :]


def int4_codes(x, group):
    """The integer codes and scales the fake quantiser rounds to (for checks)."""
    torch = _torch()
    N = x.shape[-2]
    g = x.reshape(*x.shape[:-2], -1, group * x.shape[-1]) if N % group == 0 else None
    if g is None:
        raise ValueError("token count must be a multiple of the group for int4_codes")
    amax = g.abs().amax(-1, keepdim=True)
    inv = torch.where(amax > 0, 7.0 / torch.where(amax > 0, amax, torch.ones_like(amax)), torch.zeros_like(amax))
    codes = torch.clamp(torch.round(g * inv), -7, 7).reshape(x.shape).to(torch.int8)
    scales = torch.where(amax > 0, amax / 7.0, torch.zeros_like(amax)).squeeze(-1)
    return codes, scales


@dataclass
class CalibResult:
    blocks: np.ndarray                       # float64 [D/2][2][2]: pass as rot_blocks
    angles: np.ndarray                       # float64 [D/2]
    history: list = field(default_factory=list)   # objective per step (sampled rows/cols)
    initial: float = 0.0                     # objective of the initial blocks on the evaluation sample
    final: float = 0.0                       # objective of the returned blocks on the same sample


class _Problem:
    def __init__(self, q, k, grid, split, theta, mode, q_group, k_group, device):
        torch = _torch()
        if mode not in ("interleaved", "half"):
            raise ValueError("mode must be 'interleaved' or 'half'")
        if sum(split) != D or any(s % 2 for s in split):
            raise ValueError("split must be three even widths summing to 128")
        qf, kf = _as_float(q, device), _as_float(k, device)
        if qf.dim() == 2:
            qf, kf = qf[None], kf[None]
        N = grid[0] * grid[1] * grid[2]
        if qf.shape[-2:] != (N, D) or kf.shape != qf.shape:
            raise ValueError(f"q and k must be [heads, {N}, {D}] (or [{N}, {D}])")
        cos, sin = rope_tables(grid, split, theta, device)
        yq, yk = apply_rope(qf, cos, sin), apply_rope(kf, cos, sin)
        if mode == "half":
            perm = torch.tensor(half_permutation(split), device=device)
            yq, yk = yq[..., perm], yk[..., perm]
        # smoothing (Sec. 4): per head and channel, the mean over tokens; it commutes with R
        self.qs = yq - yq.mean(-2, keepdim=True)
        self.ks = yk - yk.mean(-2, keepdim=True)
        self.q_group, self.k_group = q_group, k_group
        self.N = N

    def objective(self, R, rows, cols):
        """Mean over heads of ||Y - Q4(Q_s R) Q4(K_s R)^T||_F^2 on sampled rows/cols,
        divided by ||Y||_F^2 (so that it reads as a relative squared error)."""
        zq = fake_quant(apply_blocks(self.qs, R), self.q_group)
        zk = fake_quant(apply_blocks(self.ks, R), self.k_group)
        Y = self.qs[:, rows] @ self.ks[:, cols].transpose(-1, -2)
        Yq = zq[:, rows] @ zk[:, cols].transpose(-1, -2)
        return ((Y - Yq) ** 2).sum() / (Y ** 2).sum()


def calibrate_rotation(q, k, grid, split=(44, 42, 42), theta=10000.0, *, mode="half", q_group=1, k_group=1,
                       steps=200, lr=0.02, rows=1024, cols=2048, seed=0, init=None, kinds=None,
                       device=None) -> CalibResult:
    """Fit the angles of the O(2) blocks (Sec. 4.1.4 objective) with Adam.

    q, k: pre-RoPE calibration queries and keys of one layer, [N, 128] or
    [heads, N, 128] (bf16 bit patterns as uint16 numpy, float arrays, or float
    tensors); one rotation is fitted for all heads given.  grid/split/theta:
    the 3D RoPE.  mode: "interleaved" or "half".  q_group / k_group: tokens
    per INT4 scale (1 = per token).  init: starting angles [64] (default pi/4,
    i.e. H_2); kinds: 1 = reflection, 0 = rotation per block (default all
    reflections, the family of H_2).  Each step samples `rows` query and `cols`
    key tokens; the returned blocks are the best of the run on a fixed
    evaluation sample.
    """
    torch = _torch()
    if device is None:
        device = "cuda" if torch.cuda.is_available() else "cpu"
    prob = _Problem(q, k, grid, split, theta, mode, q_group, k_group, device)
    P = D // 2
    a0 = torch.full((P,), math.pi / 4, dtype=torch.float64) if init is None else torch.as_tensor(init, dtype=torch.float64)
    kd = torch.ones(P, dtype=torch.int64) if kinds is None else torch.as_tensor(kinds, dtype=torch.int64)
    angles = a0.clone().to(device).float().requires_grad_(True)
    kd = kd.to(device)
    gen = torch.Generator(device="cpu").manual_seed(seed)
    nr, nc = min(rows, prob.N), min(cols, prob.N)
    ev_r = torch.randperm(prob.N, generator=gen)[:nr].to(device)
    ev_c = torch.randperm(prob.N, generator=gen)[:nc].to(device)

    def evaluate(a):
        with torch.no_grad():
            return float(prob.objective(blocks_from_angles(a, kd), ev_r, ev_c))

    initial = evaluate(angles.detach())
    best, best_a = initial, angles.detach().clone()
    opt = torch.optim.Adam([angles], lr=lr)
    hist = []
    for _ in range(steps):
        r = torch.randperm(prob.N, generator=gen)[:nr].to(device)
        c = torch.randperm(prob.N, generator=gen)[:nc].to(device)
        opt.zero_grad()
        loss = prob.objective(blocks_from_angles(angles, kd), r, c)
        loss.backward()
        opt.step()
        hist.append(float(loss.detach()))
        e = evaluate(angles.detach())
        if e < best:
            best, best_a = e, angles.detach().clone()
    R = blocks_from_angles(best_a.double(), kd).cpu().numpy().astype(np.float64)
    return CalibResult(blocks=R, angles=best_a.double().cpu().numpy(), history=hist, initial=initial, final=best)
