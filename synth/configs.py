"""Seeded synthetic agent-shaped batches for the fused turn-KL path.

The paper trains on multi-turn agent rollouts (ALFWorld, WebShop, multi-hop
search); none of those datasets or models are available, so these seeded
batches stand in for them.  Each batch copies the paper's structure:
  * a batch packs trajectories back to back; trajectory b has turns
    t = 0, 1, ...; each turn is an observation span (environment text, not
    supervised) followed by the model response (supervised);
  * turn caps and counts in the range the paper uses (tens of turns);
  * survivors thin out with depth (turn counts vary per trajectory);
  * student-teacher disagreement that can decay with turn depth.

The per-token structure (trajectory ids, turn ids, loss mask, per-row teacher
noise scale) is drawn on the host with numpy's seeded PCG64.  The logits are
drawn by the counter-based generator in synth/csrc/synth.hip, on the device
for full-size batches or on the host for any subset of rows; both give the
same bits.  Nothing here computes any part of the loss.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

from . import _lib

SEED_BASE = 20260700

BF16 = "bf16"
F32 = "f32"


@dataclasses.dataclass
class Workload:
    name: str
    description: str
    vocab: int
    dtype: str
    traj_id: np.ndarray        # int32 [N], sorted, -1 = padding
    turn_id: np.ndarray        # int32 [N]
    loss_mask: np.ndarray      # uint8 [N], 1 = supervised response token
    teacher_sigma: np.ndarray  # float32 [N], standard deviation of the teacher noise per row
    seed: int
    student_sigma: float
    n_peaks: int = 0
    peak_boost: float = 0.0
    shift_prob: float = 0.0
    alphas: tuple = (0.5,)
    max_turns: int = 64
    in_place: bool = False

    @property
    def n_tokens(self) -> int:
        return int(self.traj_id.shape[0])

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == BF16 else 4

    @property
    def n_supervised(self) -> int:
        return int(self.loss_mask.sum())

    def params(self, ld: int | None = None) -> _lib.SynthParams:
        p = _lib.SynthParams()
        p.seed = self.seed
        p.vocab = self.vocab
        p.ld = self.vocab if ld is None else ld
        p.dtype = 0 if self.dtype == BF16 else 1
        p.n_peaks = self.n_peaks
        p.student_sigma = float(np.float32(self.student_sigma))
        p.peak_boost = float(np.float32(self.peak_boost))
        p.shift_threshold = int(round(self.shift_prob * 2.0 ** 32)) if self.shift_prob > 0 else 0
        p.reserved = 0
        return p

    def host_logits(self, r0: int, r1: int, n_threads: int = 0):
        """Rows [r0, r1) as host arrays (uint16 bf16 bit patterns, or float32)."""
        dt = np.uint16 if self.dtype == BF16 else np.float32
        zs = np.empty((r1 - r0, self.vocab), dtype=dt)
        zt = np.empty((r1 - r0, self.vocab), dtype=dt)
        _lib.fill_host(self.params(), self.teacher_sigma, r0, r1, zs, zt, n_threads)
        return zs, zt

    def host_rows(self, rows, n_threads: int = 0):
        """Arbitrary rows (absolute indices, any order) as host arrays."""
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        dt = np.uint16 if self.dtype == BF16 else np.float32
        zs = np.empty((rows.shape[0], self.vocab), dtype=dt)
        zt = np.empty((rows.shape[0], self.vocab), dtype=dt)
        _lib.fill_host_rows(self.params(), self.teacher_sigma, rows, zs, zt, n_threads)
        return zs, zt

    def device_logits(self, ld: int | None = None, device: str = "cuda"):
        """Full student and teacher logits generated in device memory.

        Returns (zs, zt) torch tensors of shape [N, V] (views of [N, ld]
        storage when ld > V; the padding columns are left unwritten).
        """
        import torch
        ld = self.vocab if ld is None else ld
        tdt = torch.bfloat16 if self.dtype == BF16 else torch.float32
        n = self.n_tokens
        zs = torch.empty((n, ld), dtype=tdt, device=device)
        zt = torch.empty((n, ld), dtype=tdt, device=device)
        ts = torch.from_numpy(self.teacher_sigma).to(device)
        stream = torch.cuda.current_stream().cuda_stream
        if n:
            _lib.fill_device(self.params(ld), ts.data_ptr(), 0, n, zs.data_ptr(), zt.data_ptr(),
                             stream)
        torch.cuda.current_stream().synchronize()
        del ts
        return zs[:, :self.vocab], zt[:, :self.vocab]


# ----------------------------------------------------------------------------
# structure helpers


def _obs_len(length: int, obs_frac: float) -> int:
    return int(math.floor(obs_frac * length + 0.5))


def _pack(turn_lengths: list[list[int]], obs_fracs: list[float]):
    """Pack trajectories (lists of turn lengths) with an observation prefix per turn."""
    traj, turn, mask = [], [], []
    for b, lens in enumerate(turn_lengths):
        for t, n in enumerate(lens):
            o = _obs_len(n, obs_fracs[b])
            traj.append(np.full(n, b, np.int32))
            turn.append(np.full(n, t, np.int32))
            m = np.ones(n, np.uint8)
            m[:o] = 0
            mask.append(m)
    return (np.concatenate(traj), np.concatenate(turn), np.concatenate(mask))


def _sigma(sigma) -> np.ndarray:
    return np.asarray(sigma, dtype=np.float32)


def _largest_remainder(lengths: np.ndarray, total: int, minimum: int) -> np.ndarray:
    x = lengths.astype(np.float64) * total / float(lengths.sum())
    f = np.maximum(np.floor(x).astype(np.int64), minimum)
    rem = total - int(f.sum())
    if rem > 0:
        order = np.argsort(-(x - np.floor(x)), kind="stable")
        k = 0
        while rem > 0:
            f[order[k % len(f)]] += 1
            rem -= 1
            k += 1
    while rem < 0:
        order = np.argsort(-f, kind="stable")
        for i in order:
            if rem == 0:
                break
            if f[i] > minimum:
                f[i] -= 1
                rem += 1
    assert int(f.sum()) == total and int(f.min()) >= minimum
    return f


# ----------------------------------------------------------------------------
# the five batches


def tiny() -> Workload:
    seed = SEED_BASE + 1
    rng = np.random.default_rng(seed)
    lens = [[int(v) for v in rng.integers(8, 33, size=4)] for _ in range(2)]
    traj, turn, mask = _pack(lens, [0.0, 0.0])
    return Workload(
        name="tiny", description="2 trajectories x 4 turns, turn lengths U{8..32}, V=1024 fp32",
        vocab=1024, dtype=F32, traj_id=traj, turn_id=turn, loss_mask=mask,
        teacher_sigma=np.full(traj.shape, _sigma(0.5), np.float32), seed=seed,
        student_sigma=2.0, alphas=(0.5,), max_turns=4)


def agent() -> Workload:
    seed = SEED_BASE + 2
    rng = np.random.default_rng(seed)
    lens = [[int(v) for v in rng.integers(16, 97, size=10)] for _ in range(8)]
    traj, turn, mask = _pack(lens, [0.4] * 8)
    return Workload(
        name="agent", description="8 trajectories x 10 turns, turn lengths U{16..96}, 40% observation"
        "-masked, V=32000 bf16", vocab=32000, dtype=BF16, traj_id=traj, turn_id=turn,
        loss_mask=mask, teacher_sigma=np.full(traj.shape, _sigma(1.0), np.float32), seed=seed,
        student_sigma=3.0, alphas=(0.25,), max_turns=10)


def peaked() -> Workload:
    seed = SEED_BASE + 3
    rng = np.random.default_rng(seed)
    lens = [[int(v) for v in rng.integers(8, 61, size=30)] for _ in range(16)]
    traj, turn, mask = _pack(lens, [0.6] * 16)
    return Workload(
        name="peaked", description="16 trajectories x 30 turns, turn lengths U{8..60}, 60% observation"
        "-masked, 5 peaked columns per row (+10, teacher peaks re-drawn on 20% of rows), "
        "V=151936 bf16", vocab=151936, dtype=BF16, traj_id=traj, turn_id=turn, loss_mask=mask,
        teacher_sigma=np.full(traj.shape, _sigma(1.0), np.float32), seed=seed, student_sigma=3.0,
        n_peaks=5, peak_boost=10.0, shift_prob=0.2, alphas=(0.0, 0.25, 0.5, 1.0), max_turns=30)


def long_horizon(n_tokens: int = 65536) -> Workload:
    seed = SEED_BASE + 4
    rng = np.random.default_rng(seed)
    lens: list[list[int]] = []
    total = 0
    # up to 32 trajectories, more only if they fall short of n_tokens
    while total < n_tokens:
        t_b = int(rng.integers(20, 51))
        ls = np.clip(np.rint(rng.lognormal(4.0, 0.6, size=t_b)), 4, 512).astype(np.int64)
        lens.append([int(v) for v in ls])
        total += int(ls.sum())
    # cut the packed batch at exactly n_tokens tokens
    traj, turn, mask = _pack(lens, [0.4] * len(lens))
    traj, turn, mask = traj[:n_tokens], turn[:n_tokens], mask[:n_tokens]
    sigma_t = 1.5 * np.power(0.95, turn.astype(np.float64))
    return Workload(
        name="long_horizon", description=f"{len(lens)} trajectories, turns U{{20..50}}, turn lengths "
        f"lognormal(4, 0.6) clipped to [4, 512], cut at {n_tokens} tokens, 40% observation-masked, "
        "teacher noise 1.5*0.95^turn, V=151936 bf16", vocab=151936, dtype=BF16, traj_id=traj,
        turn_id=turn, loss_mask=mask, teacher_sigma=_sigma(sigma_t), seed=seed, student_sigma=3.0,
        alphas=(0.5,), max_turns=50)


def stress(n_tokens: int = 131072) -> Workload:
    seed = SEED_BASE + 5
    rng = np.random.default_rng(seed)
    n_traj = 64
    k = np.arange(1, 201, dtype=np.float64)
    p = k ** -1.3
    p /= p.sum()
    t_b = rng.choice(np.arange(1, 201), size=n_traj, p=p)
    t_b[0] = max(int(t_b[0]), 2)  # trajectory 0 carries one fully masked turn
    raw = [np.clip(np.rint(rng.lognormal(4.0, 0.6, size=int(t))), 4, 512).astype(np.int64)
           for t in t_b]
    flat = _largest_remainder(np.concatenate(raw), n_tokens, 4)
    lens, o = [], 0
    for r in raw:
        lens.append([int(v) for v in flat[o:o + len(r)]])
        o += len(r)
    modes = rng.integers(0, 4, size=n_traj)  # 0 all ones, 1 40% obs, 2 60% obs, 3 Bernoulli(0.5)
    fracs = [{0: 0.0, 1: 0.4, 2: 0.6, 3: 0.0}[int(m)] for m in modes]
    traj, turn, mask = _pack(lens, fracs)
    for b in range(n_traj):
        if modes[b] == 3:
            sel = traj == b
            mask[sel] = rng.integers(0, 2, size=int(sel.sum())).astype(np.uint8)
    mask[(traj == 0) & (turn == 1)] = 0
    mask[traj == n_traj - 1] = 0
    return Workload(
        name="stress", description=f"{n_tokens} tokens over 64 trajectories, turn counts Zipf(1.3) on "
        "{1..200}, lognormal turn lengths rescaled to the total, mixed masks (one fully masked turn, "
        "one fully masked trajectory), V=151936 bf16, gradient written in place", vocab=151936,
        dtype=BF16, traj_id=traj, turn_id=turn, loss_mask=mask,
        teacher_sigma=np.full(traj.shape, _sigma(1.0), np.float32), seed=seed, student_sigma=3.0,
        alphas=(0.75,), max_turns=200, in_place=True)


WORKLOADS = {"tiny": tiny, "agent": agent, "peaked": peaked, "long_horizon": long_horizon,
             "stress": stress}


def make(name: str, **kw) -> Workload:
    return WORKLOADS[name](**kw)
