"""Helpers for the GPU parity tests: run the HIP path through the C ABI, run
the CPU oracle on the same seeded inputs, and compare.

Tolerances (derived from the fp32 arithmetic of the kernels):
  * segment table, counts, survivors, status codes: bit-exact;
  * loss (each of L_blend, L_traj, L_turn): relative 1e-4, with an absolute
    floor of 1e-6 (each per-token KL carries ~1e-7 absolute error from the
    fp32 exp2 / log2 of the row scalars, visible only when KL is ~0);
  * per-token KL: |d| <= 2e-4 |KL| + 5e-6;
  * gradient, compared unweighted (g_hat = G / (grad_scale * w_i)):
      |g_hat - g| <= 2e-2 absolute (the stated bar), and the tighter
      |g_hat - g| <= 2^-8 |g| + 2e-5 for bf16 output (about one bf16 ulp),
      |g_hat - g| <= 1e-4 |g| + 2e-6 for fp32 output;
    unsupervised rows must be exactly zero;
  * per-turn stats: mean and loss mass relative 1e-4 (absolute floor 1e-6),
    variance |d| <= 1e-4 var + 1e-8.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_device_logits(arr: np.ndarray, device="cuda") -> torch.Tensor:
    """Host logits (uint16 bf16 patterns or float32) -> device tensor."""
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(arr).to(device)


def rows_to_host(t: torch.Tensor, rows) -> np.ndarray:
    """Selected rows of a device bf16/fp32 matrix as float32 on the host."""
    idx = torch.as_tensor(np.asarray(rows, np.int64), device=t.device)
    sel = t.index_select(0, idx)
    if sel.dtype == torch.bfloat16:
        u = sel.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return (u.astype(np.uint32) << 16).view(np.float32)
    return sel.float().cpu().numpy()


def oracle_dtype(dtype: torch.dtype) -> int:
    return O.DTYPE_BF16 if dtype == torch.bfloat16 else O.DTYPE_F32


def ids_to_device(traj, turn, mask, device="cuda"):
    return (torch.from_numpy(np.ascontiguousarray(turn, np.int32)).to(device),
            torch.from_numpy(np.ascontiguousarray(traj, np.int32)).to(device),
            torch.from_numpy(np.ascontiguousarray(mask, np.uint8)).to(device))


def check_segments(ws: T.Workspace, ref: O.Segments) -> None:
    got = ws.segments()
    assert len(got["start"]) == ref.count, (len(got["start"]), ref.count)
    for k in ("start", "length", "traj", "turn", "n_sup"):
        assert np.array_equal(got[k], getattr(ref, k)), k


def check_loss(loss: torch.Tensor, ref_loss, rtol=1e-4) -> None:
    got = loss.cpu().numpy().astype(np.float64)
    for g, r, name in zip(got, ref_loss, ("L_blend", "L_traj", "L_turn")):
        assert abs(g - r) <= rtol * abs(r) + 1e-6, (name, g, r, abs(g - r) / max(abs(r), 1e-30))


def check_token_kl(kl_dev: torch.Tensor, ref_kl: np.ndarray, mask: np.ndarray) -> None:
    got = kl_dev.cpu().numpy()[: ref_kl.shape[0]].astype(np.float64)
    err = np.abs(got - ref_kl)
    bound = 2e-4 * np.abs(ref_kl) + 5e-6
    bad = np.nonzero(err > bound)[0]
    assert bad.size == 0, (bad[:5], got[bad[:5]], ref_kl[bad[:5]])
    assert np.all(got[np.asarray(mask) == 0] == 0.0)


def check_token_weights(w_dev: torch.Tensor, ref_w: np.ndarray, mask: np.ndarray) -> None:
    """w_i is the fp64 weight rounded to float: within one float rounding of
    the oracle's value, exactly 0 for unsupervised tokens."""
    got = w_dev.cpu().numpy()[: ref_w.shape[0]].astype(np.float64)
    err = np.abs(got - ref_w)
    bad = np.nonzero(err > 2.0 ** -23 * np.abs(ref_w))[0]
    assert bad.size == 0, (bad[:5], got[bad[:5]], ref_w[bad[:5]])
    assert np.all(got[np.asarray(mask) == 0] == 0.0)


def check_token_lse(lse_dev: torch.Tensor, ref_lse: np.ndarray, mask: np.ndarray) -> None:
    """Log-partition functions of supervised rows within 2e-5 + 1e-6 |lse| of
    the oracle's float64 values (float references and sums); NaN for
    unsupervised rows, which are never read."""
    n = ref_lse.shape[0]
    got = lse_dev.reshape(-1)[: 2 * n].reshape(n, 2).cpu().numpy().astype(np.float64)
    sup = np.asarray(mask)[:n] != 0
    assert np.all(np.isnan(got[~sup]))
    err = np.abs(got[sup] - ref_lse[sup])
    bound = 2e-5 + 1e-6 * np.abs(ref_lse[sup])
    bad = np.argwhere(err > bound)
    assert bad.size == 0, (bad[:5], got[sup][tuple(bad[:5].T)], ref_lse[sup][tuple(bad[:5].T)])


def check_stats(stats_buf: torch.Tensor, ref: np.ndarray) -> None:
    got = T.read_turn_stats(stats_buf)
    assert np.array_equal(got["n_tokens"], ref["n_tokens"])
    assert np.array_equal(got["n_traj"], ref["n_traj"])
    for f in ("kl_mean", "loss_mass"):
        err = np.abs(got[f] - ref[f])
        assert np.all(err <= 1e-4 * np.abs(ref[f]) + 1e-6), (f, np.max(err))
    err = np.abs(got["kl_var"] - ref["kl_var"])
    assert np.all(err <= 1e-4 * ref["kl_var"] + 1e-8), ("kl_var", np.max(err))
    err = np.abs(got["kl_m2"] - ref["kl_m2"])
    assert np.all(err <= 1e-4 * ref["kl_m2"] + 1e-8 * np.maximum(ref["n_tokens"], 1)), \
        ("kl_m2", np.max(err))


def check_grad_rows(grad_dev: torch.Tensor, ref: O.Result, grad_scale: float, rows,
                    mask: np.ndarray) -> float:
    """Compare gradient rows; returns the worst unweighted absolute error."""
    rows = list(rows)
    G = rows_to_host(grad_dev, rows).astype(np.float64)
    bf16 = grad_dev.dtype == torch.bfloat16
    worst = 0.0
    for k, r in enumerate(rows):
        if not mask[r]:
            assert np.all(G[k] == 0.0), ("unsupervised row not zero", r)
            continue
        g_ref = ref.grads[r]
        scale = grad_scale * ref.w[r]
        if scale == 0.0:  # a supervised token of weight 0 (a turn below the support floor)
            assert np.all(G[k] == 0.0), ("zero-weight row not zero", r)
            continue
        g_hat = G[k] / scale
        err = np.abs(g_hat - g_ref)
        worst = max(worst, float(err.max()))
        assert err.max() <= 2e-2, (r, err.max())
        bound = (2.0 ** -8 * np.abs(g_ref) + 2e-5) if bf16 else (1e-4 * np.abs(g_ref) + 2e-6)
        bad = np.nonzero(err > bound)[0]
        assert bad.size == 0, (r, bad[:5], g_hat[bad[:5]], g_ref[bad[:5]])
    return worst


def sample_rows(mask: np.ndarray, n_sup: int = 24, n_unsup: int = 4, seed: int = 0):
    """First, last and random supervised rows, plus a few unsupervised ones."""
    rng = np.random.default_rng(seed)
    sup = np.nonzero(mask)[0]
    uns = np.nonzero(np.asarray(mask) == 0)[0]
    pick = set()
    if sup.size:
        pick |= {int(sup[0]), int(sup[-1])}
        pick |= set(int(x) for x in rng.choice(sup, size=min(n_sup, sup.size), replace=False))
    if uns.size:
        pick |= set(int(x) for x in rng.choice(uns, size=min(n_unsup, uns.size), replace=False))
    return sorted(pick)


def rows_bits_to_host(t: torch.Tensor, rows) -> np.ndarray:
    """Selected rows of a device matrix in the oracle's input format
    (uint16 bf16 patterns, or float32)."""
    idx = torch.as_tensor(np.asarray(rows, np.int64), device=t.device)
    sel = t.index_select(0, idx).contiguous()
    if sel.dtype == torch.bfloat16:
        return sel.view(torch.int16).cpu().numpy().view(np.uint16)
    return sel.cpu().numpy()


def device_row_source(zs: torch.Tensor, zt: torch.Tensor):
    """Oracle row source reading the generator's output from device memory."""
    return lambda rows: (rows_bits_to_host(zs, rows), rows_bits_to_host(zt, rows))


def ticket_order_rows(mask: np.ndarray, n_ends: int = 100, n_random: int = 800, seed: int = 0):
    """Supervised rows for a full-size gradient comparison: the first and the
    last n_ends supervised rows (the two ends of the row kernel's row-major
    ticket order) and n_random others.  Every row covers all of its chunks."""
    rng = np.random.default_rng(seed)
    sup = np.nonzero(np.asarray(mask))[0]
    pick = set(int(x) for x in sup[:n_ends]) | set(int(x) for x in sup[-n_ends:])
    rest = np.setdiff1d(sup, np.fromiter(pick, np.int64, len(pick)))
    if rest.size:
        pick |= set(int(x) for x in rng.choice(rest, size=min(n_random, rest.size), replace=False))
    return sorted(pick)


def check_grad_rows_batched(grad_dev: torch.Tensor, w: np.ndarray, grad_scale: float, rows,
                            host_rows, dtype: int, batch: int = 128) -> float:
    """check_grad_rows on many rows with bounded host memory: the oracle's
    unweighted row gradients are computed batch by batch from host copies of
    the logit rows, host_rows(rows) -> (zs, zt), and compared with the device
    rows.  Returns the worst unweighted absolute error."""
    rows = np.asarray(sorted(rows), np.int64)
    worst = 0.0
    bf16 = grad_dev.dtype == torch.bfloat16
    for k0 in range(0, rows.shape[0], batch):
        r = rows[k0:k0 + batch]
        zs, zt = host_rows(r)
        _, g_ref = O.row_kl(zs, zt, dtype, want_grad=True)
        G = rows_to_host(grad_dev, r).astype(np.float64)
        scale = grad_scale * np.asarray(w)[r]
        assert np.all(scale != 0.0)
        err = np.abs(G / scale[:, None] - g_ref)
        worst = max(worst, float(err.max()))
        assert err.max() <= 2e-2, (k0, err.max())
        bound = (2.0 ** -8 * np.abs(g_ref) + 2e-5) if bf16 else (1e-4 * np.abs(g_ref) + 2e-6)
        bad = np.argwhere(err > bound)
        assert bad.size == 0, (r[bad[:5, 0]], bad[:5, 1], err[tuple(bad[:5].T)])
    return worst


def check_grad_every_row_on_device(grad_dev: torch.Tensor, mask: np.ndarray, w: np.ndarray,
                                   grad_scale: float, block: int = 4096) -> None:
    """Properties every gradient row must have, checked on the device over
    all rows in blocks: each unsupervised row is exactly zero (in place, that
    proves the row's student logits were overwritten), and each supervised
    row sums to zero, as dKL/dz_s does (sum_v p_s(v) (d_v - KL) = 0), up to
    the rounding of its stored elements: |sum_v G| <= 2^-8 sum_v |G| +
    1e-6 |grad_scale w_i|."""
    dev = grad_dev.device
    mask = np.asarray(mask)
    uns = np.nonzero(mask == 0)[0]
    for k0 in range(0, uns.shape[0], block):
        idx = torch.from_numpy(uns[k0:k0 + block]).to(dev)
        nz = int(torch.count_nonzero(grad_dev.index_select(0, idx)).item())
        assert nz == 0, ("unsupervised rows with nonzero gradient", k0, nz)
    sup = np.nonzero(mask)[0]
    for k0 in range(0, sup.shape[0], block):
        r = sup[k0:k0 + block]
        g = grad_dev.index_select(0, torch.from_numpy(r).to(dev)).float()
        s = g.sum(dim=1).double().cpu().numpy()
        a = g.abs().sum(dim=1).double().cpu().numpy()
        del g
        floor = 1e-6 * np.abs(grad_scale * np.asarray(w)[r])
        bad = np.nonzero(np.abs(s) > 2.0 ** -8 * a + floor)[0]
        assert bad.size == 0, ("row sums", r[bad[:5]], s[bad[:5]], a[bad[:5]])
