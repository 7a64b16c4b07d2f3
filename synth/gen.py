"""Seeded draws: gradients g_t^(m) for every worker m and iteration t, and the
initial parameters w_0.  Rows have stride ld; the padding [d, ld) is zero.

Gradient law per group of the workload: N(0, sigma^2) or Laplace(0, b).
Parameters: w_0 ~ N(0, 0.02^2).
"""
import numpy as np

_MIX = 0x9E3779B97F4A7C15


def _stream_seed(seed, t, salt=0):
    return (seed * 1_000_003 + t * 7919 + salt * 104_729) & ((1 << 63) - 1)


def _scale_vector_np(w):
    s = np.zeros(w.d, np.float32)
    for (a, b), sc in zip(w.groups, w.group_scale):
        s[a:b] = sc
    return s


def gradients_np(w, t, rows=None):
    """numpy draw of the [M][ld] float32 gradient batch of iteration t (or of
    the listed rows only; each row has its own stream, so a subset equals the
    same rows of the full batch)."""
    rows = range(w.M) if rows is None else rows
    out = np.zeros((len(rows), w.ld), np.float32)
    sv = _scale_vector_np(w)
    for r, m in enumerate(rows):
        rng = np.random.default_rng(_stream_seed(w.seed, t, 1 + m))
        if w.law == "laplace":
            x = rng.laplace(0.0, 1.0, size=w.d).astype(np.float32)
        else:
            x = rng.standard_normal(size=w.d, dtype=np.float32)
        out[r, :w.d] = x * sv
    return out


def init_params_np(w):
    rng = np.random.default_rng(_stream_seed(w.init_seed, 0))
    out = np.zeros(w.ld, np.float32)
    out[:w.d] = rng.standard_normal(size=w.d, dtype=np.float32) * np.float32(0.02)
    return out


def gradients(w, t, device="cuda", out=None):
    """torch draw of the [M][ld] float32 gradient batch of iteration t on
    `device` (written into `out` if given).  Deterministic for a given device
    type; the tests copy the very same bytes to the oracle."""
    import torch
    if out is None:
        out = torch.empty((w.M, w.ld), dtype=torch.float32, device=device)
    gen = torch.Generator(device=out.device)
    gen.manual_seed(_stream_seed(w.seed, t))
    body = out[:, :w.d]
    if w.law == "laplace":
        body.uniform_(-0.5, 0.5, generator=gen)
        a = body.abs().clamp_(max=0.5 - 2.0 ** -25)
        body.copy_(-torch.sign(body) * torch.log1p(-2.0 * a))
        del a
    else:
        body.normal_(0.0, 1.0, generator=gen)
    sv = torch.from_numpy(_scale_vector_np(w)).to(out.device)
    body.mul_(sv)
    if w.ld > w.d:
        out[:, w.d:].zero_()
    return out


def init_params(w, device="cuda"):
    import torch
    return torch.from_numpy(init_params_np(w)).to(device)
