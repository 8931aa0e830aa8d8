"""Edge cases, tilings, error paths and invariants of the HIP path, each
checked against the CPU oracle (or an exact property) through the C ABI."""
import numpy as np
import pytest
import torch

from gpu_support import (check_grad_rows, check_loss, check_segments, check_stats,
                         check_token_kl, check_token_lse, check_token_weights, ids_to_device, log,
                         to_device_logits)
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T

pytestmark = pytest.mark.gpu


def bf16_bits(x):
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def make_batch(seed, n_traj=5, max_turns=6, V=1000, dtype="bf16", pad=True, sigma=3.0,
               noise=1.0, min_len=1, max_len=40):
    rng = np.random.default_rng(seed)
    traj, turn, mask = [], [], []
    for b in range(n_traj):
        turns = np.sort(rng.choice(max_turns, size=int(rng.integers(1, max_turns + 1)),
                                   replace=False))
        for t in turns:
            n = int(rng.integers(min_len, max_len + 1))
            if pad and rng.uniform() < 0.2:
                k = int(rng.integers(1, 4))
                traj += [-1] * k
                turn += [0] * k
                mask += [0] * k
            traj += [b] * n
            turn += [int(t)] * n
            mode = int(rng.integers(0, 4))
            if mode == 0:
                mask += [0] * n
            elif mode == 1:
                mask += [1] * n
            else:
                o = n * 2 // 5
                mask += [0] * o + [1] * (n - o)
    traj = np.array(traj, np.int32)
    turn = np.array(turn, np.int32)
    mask = np.array(mask, np.uint8)
    zs = rng.normal(0.0, sigma, (len(traj), V)).astype(np.float32)
    zt = (zs + rng.normal(0.0, noise, zs.shape)).astype(np.float32)
    if dtype == "bf16":
        zs, zt = bf16_bits(zs), bf16_bits(zt)
    return traj, turn, mask, zs, zt


def run_both(traj, turn, mask, zs_h, zt_h, alpha=0.4, max_turns=8, grad_scale=1.0, ld=None,
             grad="new", grad_rows=None, vpt=0):
    dev = "cuda"
    n, V = zs_h.shape
    if ld is None:
        zs, zt = to_device_logits(zs_h, dev), to_device_logits(zt_h, dev)
    else:  # padded row stride; the padding holds NaN and must never be read
        def padded(h):
            full = np.full((n, ld), np.nan, np.float32)
            d = to_device_logits(full.astype(np.float32), dev)
            if h.dtype == np.uint16:
                d = d.to(torch.bfloat16)
            d[:, :V] = to_device_logits(h, dev)
            return d[:, :V]
        zs, zt = padded(zs_h), padded(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask, dev)
    stats = T.new_turn_stats(max_turns)
    T.set_row_tiling(vpt)
    try:
        loss, g, _, kl, ws = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, alpha, grad_scale=grad_scale,
                                       grad=grad, max_turns=max_turns, turn_stats=stats,
                                       token_kl=True)
    finally:
        T.set_row_tiling(0)
    torch.cuda.synchronize()
    rows = list(range(n)) if grad_rows is None else grad_rows
    dt = O.DTYPE_BF16 if zs_h.dtype == np.uint16 else O.DTYPE_F32
    ref = O.fwd_bwd(traj, turn, mask, alpha, max_turns, lambda r: (zs_h[r], zt_h[r]), dt,
                    grad_scale, rows)
    return (loss, g, stats, kl, ws), ref, rows


def check_all(out, ref, mask, grad_scale, rows):
    loss, g, stats, kl, ws = out
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, mask)
    check_stats(stats, ref.stats)
    if g is not None:
        check_grad_rows(g, ref, grad_scale, rows, mask)


# ----------------------------------------------------------------------------
# tilings and vocabulary shapes


@pytest.mark.parametrize("V,dtype,vpt", [
    (1024, "f32", 0), (1024, "f32", 1),            # one chunk / four chunks per row
    (32000, "bf16", 0), (32000, "bf16", 1), (32000, "bf16", 3), (32000, "bf16", 7),
    (4096, "bf16", 1), (12296, "bf16", 2), (40000, "f32", 5),
    # chunk boundaries on 1 KiB multiples (32000 x 2), on 128-byte multiples
    # (4392 x 2: the 1 KiB rounding would leave a chunk too short), and balanced
    # (8240 x 3: neither rounding keeps every chunk long enough)
    (32000, "bf16", 2), (4392, "bf16", 2), (8240, "bf16", 3),
])
def test_tilings(V, dtype, vpt, gpu):
    log(f"tiling V={V} {dtype} vpt={vpt}")
    traj, turn, mask, zs, zt = make_batch(V + vpt, V=V, dtype=dtype)
    out, ref, rows = run_both(traj, turn, mask, zs, zt, vpt=vpt)
    check_all(out, ref, mask, 1.0, rows)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_full_vocabulary_default_tiling(dtype, gpu):
    """V = 151,936 with the default tiling: 3 chunks (bf16) or 6 chunks (fp32)
    with 1 KiB-aligned boundaries, every row and gradient checked."""
    log(f"V=151936 {dtype} default tiling")
    traj, turn, mask, zs, zt = make_batch(77, n_traj=3, max_turns=4, V=151936, dtype=dtype,
                                          max_len=12)
    out, ref, rows = run_both(traj, turn, mask, zs, zt)
    check_all(out, ref, mask, 1.0, rows)


@pytest.mark.parametrize("share", [1.0, 0.9, 0.89, 0.5])
def test_both_load_orders(share, gpu):
    """The bf16 row kernel runs in one of two load orders, chosen on the device
    from the supervised share of the rows (alternating above 90%, split
    otherwise); both give the oracle's results at the default tiling."""
    log(f"load order, supervised share {share}")
    traj, turn, mask, zs, zt = make_batch(95, n_traj=4, max_turns=5, V=151936, dtype="bf16",
                                          pad=False, min_len=5, max_len=10)
    n = len(traj)
    k = int(round(share * n))
    mask = np.zeros(n, np.uint8)
    mask[np.random.default_rng(3).permutation(n)[:k]] = 1
    out, ref, rows = run_both(traj, turn, mask, zs, zt)
    check_all(out, ref, mask, 1.0, rows)


@pytest.mark.parametrize("V,dtype", [(6553600, "bf16"), (3276800, "f32"), (1048575, "bf16")])
def test_vocabularies_at_the_chunk_limit(V, dtype, gpu):
    """The widest rows the host accepts: 128 chunks per row, on the vector path
    (25 packs per thread, bf16 and fp32) and on the scalar path (an odd
    vocabulary, 32 elements per thread); one more pack or element is rejected
    on the host."""
    log(f"chunk limit V={V} {dtype}")
    traj, turn, mask, zs, zt = make_batch(V % 1000, n_traj=2, max_turns=2, V=V, dtype=dtype,
                                          pad=False, min_len=2, max_len=4)
    out, ref, rows = run_both(traj, turn, mask, zs, zt, max_turns=2)
    check_all(out, ref, mask, 1.0, rows)


@pytest.mark.parametrize("V,dtype", [(1, "bf16"), (7, "f32"), (24, "bf16"), (1001, "bf16"),
                                     (1003, "f32"), (50257, "bf16"), (8200, "f32")])
def test_ragged_vocabularies(V, dtype, gpu):
    """Vocabularies that are not a multiple of the 16-byte vector take the
    scalar path; tiny ones leave most lanes of a chunk idle."""
    log(f"ragged V={V} {dtype}")
    traj, turn, mask, zs, zt = make_batch(V, V=V, dtype=dtype, n_traj=3)
    out, ref, rows = run_both(traj, turn, mask, zs, zt)
    check_all(out, ref, mask, 1.0, rows)


@pytest.mark.parametrize("V,ld,dtype", [(2048, 2056, "bf16"), (2048, 2051, "bf16"),
                                        (1000, 1004, "f32"), (1000, 1001, "f32")])
def test_padded_row_stride(V, ld, dtype, gpu):
    log(f"ld V={V} ld={ld} {dtype}")
    traj, turn, mask, zs, zt = make_batch(ld, V=V, dtype=dtype)
    out, ref, rows = run_both(traj, turn, mask, zs, zt, ld=ld)
    check_all(out, ref, mask, 1.0, rows)
    assert torch.isfinite(out[0]).all()


# ----------------------------------------------------------------------------
# options


@pytest.mark.parametrize("grad_scale", [-2.5, 0.0, 1e-3])
def test_grad_scale(grad_scale, gpu):
    traj, turn, mask, zs, zt = make_batch(11)
    out, ref, rows = run_both(traj, turn, mask, zs, zt, grad_scale=grad_scale)
    if grad_scale == 0.0:
        check_all(out[:1] + (None,) + out[2:], ref, mask, 1.0, rows)
        assert torch.count_nonzero(out[1].float()).item() == 0
    else:
        check_all(out, ref, mask, grad_scale, rows)


@pytest.mark.parametrize("V,dtype,vpt,shift,grad,floor", [
    (32000, "bf16", 3, 0.0, "new", 2),      # six chunks per row, support floor
    (151936, "bf16", 0, 0.0, "inplace", 0),  # three 1 KiB-aligned chunks, in place
    (1001, "f32", 0, 0.0, None, 0),          # scalar path, forward only
    (4096, "f32", 0, 5000.0, "new", 0),      # offset chunks (|logits| > 64)
    (8240, "bf16", 3, -96.0, "new", 8),      # balanced chunks, offset rows, floor
])
def test_per_token_weights_and_log_partition_functions(V, dtype, vpt, shift, grad, floor, gpu):
    """The optional per-token outputs: w_i and both rows' log-partition
    functions (NaN for unsupervised rows), against the oracle; the other
    outputs are unchanged by asking for them."""
    log(f"per-token outputs V={V} {dtype} vpt={vpt} shift={shift} grad={grad} floor={floor}")
    traj, turn, mask, zs_h, zt_h = make_batch(300 + V % 97, n_traj=4, max_turns=5, V=V,
                                              dtype="f32", max_len=12)
    zs_h, zt_h = _as(dtype, zs_h + shift), _as(dtype, zt_h + shift * 0.5)
    n = len(traj)
    zs_copy, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    wts = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.zeros((n, 2), dtype=torch.float32, device="cuda")
    outs = []
    T.set_row_tiling(vpt)
    try:
        for extra in (dict(token_weights=wts, token_lse=lse), {}):
            stats = T.new_turn_stats(5)
            src = zs_copy.clone()
            loss, g, _, kl, ws = T.fwd_bwd(src, zt, turn_d, traj_d, mask_d, 0.4, grad=grad,
                                           max_turns=5, turn_stats=stats, token_kl=True,
                                           support_floor=floor, **extra)
            torch.cuda.synchronize()
            outs.append((loss.cpu(), None if g is None else g.cpu(), stats.cpu(), kl.cpu()))
    finally:
        T.set_row_tiling(0)
    ref = O.fwd_bwd(traj, turn, mask, 0.4, 5, lambda r: (zs_h[r], zt_h[r]),
                    O.DTYPE_BF16 if dtype == "bf16" else O.DTYPE_F32, 1.0,
                    list(range(n)), support_floor=floor)
    check_token_weights(wts, ref.w, mask)
    check_token_lse(lse, ref.lse, mask)
    check_loss(outs[0][0], ref.loss)
    check_token_kl(outs[0][3], ref.kl, mask)
    if grad is not None:
        check_grad_rows(outs[0][1], ref, 1.0, list(range(n)), mask)
    # bit-identical with and without the extra outputs
    for a, b in zip(outs[0], outs[1]):
        if a is not None:
            assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.uint8) if b.dtype == torch.bfloat16 else b)


def test_forward_only(gpu):
    traj, turn, mask, zs, zt = make_batch(12)
    out, ref, rows = run_both(traj, turn, mask, zs, zt, grad=None)
    assert out[1] is None
    check_all(out, ref, mask, 1.0, rows)


def test_in_place_equals_out_of_place_bitwise(gpu):
    traj, turn, mask, zs_h, zt_h = make_batch(13, V=32000)
    zs = to_device_logits(zs_h)
    zt = to_device_logits(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    l1, g1, _, k1, _ = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.3, max_turns=8, token_kl=True)
    zs2 = zs.clone()
    l2, g2, _, k2, _ = T.fwd_bwd(zs2, zt, turn_d, traj_d, mask_d, 0.3, max_turns=8, grad="inplace",
                                 token_kl=True)
    torch.cuda.synchronize()
    assert g2.data_ptr() == zs2.data_ptr()
    assert torch.equal(g1.view(torch.int16), zs2.view(torch.int16))
    assert torch.equal(l1, l2) and torch.equal(k1, k2)


def test_runs_are_bitwise_deterministic(gpu):
    traj, turn, mask, zs_h, zt_h = make_batch(14, V=151936 // 4, n_traj=6)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    outs = []
    for _ in range(3):
        st = T.new_turn_stats(8)
        T.set_row_tiling(2)  # several chunks per row: exercises the exchange
        try:
            l, g, _, k, _ = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.6, max_turns=8,
                                      turn_stats=st, token_kl=True)
        finally:
            T.set_row_tiling(0)
        outs.append((l, g, st, k))
    torch.cuda.synchronize()
    for l, g, st, k in outs[1:]:
        assert torch.equal(l, outs[0][0]) and torch.equal(k, outs[0][3])
        assert torch.equal(g.view(torch.int16), outs[0][1].view(torch.int16))
        assert torch.equal(st, outs[0][2])


@pytest.mark.parametrize("V,vpt,all_supervised", [(37984, 2, False), (37984, 2, True),
                                                   (151936, 0, False), (151936, 0, True)])
def test_exchange_stress_loop(V, vpt, all_supervised, gpu):
    """250 calls in a row (1,000 over the four cases) of a batch whose rows are
    split over several workgroups (10 chunks per row at V = 37,984 with 2 packs
    per thread, 3 at full width), each compared bit for bit with the first
    call on the device: loss, per-token KL, statistics and gradient.  A mixed
    batch runs the split load order, an all-supervised one the alternating
    order.  The first call is checked against the oracle."""
    traj, turn, mask, zs_h, zt_h = make_batch(15 + V % 7, V=V, n_traj=5, max_len=30)
    if all_supervised:
        mask = (traj >= 0).astype(np.uint8)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    n = len(traj)
    log(f"exchange stress: N={n} V={V} vpt={vpt} all_supervised={all_supervised}")
    T.set_row_tiling(vpt)
    try:
        ws = T.Workspace(n, V, T.BF16, 8)
        grad = torch.empty_like(zs)
        kl = torch.empty(n, dtype=torch.float32, device=gpu)
        st = T.new_turn_stats(8)
        loss, *_ = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.6, grad=grad, max_turns=8,
                             turn_stats=st, token_kl=kl, workspace=ws)
        ref = (loss.clone(), grad.clone(), kl.clone(), st.clone())
        bad = torch.zeros(4, dtype=torch.int64, device=gpu)
        for _ in range(250):
            loss, *_ = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.6, grad=grad, max_turns=8,
                                 turn_stats=st, token_kl=kl, workspace=ws, check=False)
            bad[0] += (loss != ref[0]).sum()
            bad[1] += (grad.view(torch.int16) != ref[1].view(torch.int16)).sum()
            bad[2] += (kl.view(torch.int32) != ref[2].view(torch.int32)).sum()
            bad[3] += (st != ref[3]).sum()
        torch.cuda.synchronize()
        assert ws.status() == T.OK
    finally:
        T.set_row_tiling(0)
    assert bad.tolist() == [0, 0, 0, 0]
    o = O.fwd_bwd(traj, turn, mask, 0.6, 8, lambda r: (zs_h[r], zt_h[r]), O.DTYPE_BF16, 1.0,
                  list(range(0, n, 7)))
    check_loss(ref[0], o.loss)
    check_token_kl(ref[2], o.kl, mask)
    check_stats(ref[3], o.stats)
    check_grad_rows(ref[1], o, 1.0, list(range(0, n, 7)), mask)


def test_accumulated_stats_equal_pooled_oracle(gpu):
    """Three micro-batches accumulated on the device equal the oracle's
    statistics recomputed from the pooled tokens (no merge formula)."""
    stats = T.new_turn_stats(8)
    parts = []
    for k in range(3):
        traj, turn, mask, zs_h, zt_h = make_batch(20 + k, V=3000)
        zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
        turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
        T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.5, grad=None, max_turns=8, turn_stats=stats,
                  accumulate_stats=k > 0)
        ref = O.fwd_bwd(traj, turn, mask, 0.5, 8, lambda r: (zs_h[r], zt_h[r]), O.DTYPE_BF16)
        parts.append((ref.seg, mask, ref.kl, ref.w))
    torch.cuda.synchronize()
    check_stats(stats, O.turn_stats(parts, 8))


def test_loss_is_affine_in_alpha_and_mass_sums_to_loss(gpu):
    traj, turn, mask, zs_h, zt_h = make_batch(30, V=5000)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    res = {}
    for a in (0.0, 0.35, 1.0):
        st = T.new_turn_stats(8)
        l, _, _, _, _ = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, a, grad=None, max_turns=8,
                                  turn_stats=st)
        res[a] = (l.cpu().numpy().astype(np.float64), T.read_turn_stats(st))
    for a, (l, st) in res.items():
        assert abs(l[0] - ((1 - a) * l[1] + a * l[2])) <= 1e-6 * abs(l[0])
        assert abs(st["loss_mass"].sum() - l[0]) <= 1e-6 * abs(l[0])
        assert np.allclose(l[1:], res[0.0][0][1:], rtol=0, atol=0)
    assert abs(res[0.0][0][0] - res[0.0][0][1]) <= 1e-7 * res[0.0][0][1]
    assert abs(res[1.0][0][0] - res[1.0][0][2]) <= 1e-7 * res[1.0][0][2]


# ----------------------------------------------------------------------------
# degenerate batches


def test_identical_logits_give_exact_zeros(gpu):
    traj, turn, mask, zs_h, _ = make_batch(40, V=32000)
    zs = to_device_logits(zs_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    for vpt in (0, 2):
        T.set_row_tiling(vpt)
        try:
            l, g, _, k, _ = T.fwd_bwd(zs, zs, turn_d, traj_d, mask_d, 0.5, max_turns=8,
                                      token_kl=True)
        finally:
            T.set_row_tiling(0)
        torch.cuda.synchronize()
        assert torch.count_nonzero(l).item() == 0
        assert torch.count_nonzero(k).item() == 0
        assert torch.count_nonzero(g.float()).item() == 0


def test_empty_batch(gpu):
    e = torch.empty((0, 128), dtype=torch.bfloat16, device=gpu)
    i = torch.empty(0, dtype=torch.int32, device=gpu)
    m = torch.empty(0, dtype=torch.uint8, device=gpu)
    st = T.new_turn_stats(4)
    st.fill_(7)
    l, g, _, _, _ = T.fwd_bwd(e, e.clone(), i, i.clone(), m, 0.5, max_turns=4, turn_stats=st,
                              accumulate_stats=True)
    torch.cuda.synchronize()
    assert torch.count_nonzero(l).item() == 0
    assert torch.all(st == 7)  # accumulating an empty batch changes nothing
    l, g, _, _, _ = T.fwd_bwd(e, e.clone(), i, i.clone(), m, 0.5, max_turns=4, turn_stats=st)
    torch.cuda.synchronize()
    assert torch.count_nonzero(st).item() == 0


def test_fully_masked_batch(gpu):
    traj, turn, mask, zs, zt = make_batch(41)
    mask[:] = 0
    out, ref, rows = run_both(traj, turn, mask, zs, zt)
    assert ref.loss == (0.0, 0.0, 0.0)
    check_all(out, ref, mask, 1.0, rows)
    assert torch.count_nonzero(out[1].float()).item() == 0


def test_single_giant_segment_and_one_token_segments(gpu):
    rng = np.random.default_rng(42)
    V = 512
    # one trajectory, one turn of 3000 tokens
    n = 3000
    traj = np.zeros(n, np.int32)
    turn = np.zeros(n, np.int32)
    mask = (rng.uniform(size=n) < 0.7).astype(np.uint8)
    zs = bf16_bits(rng.normal(0, 3, (n, V)))
    zt = bf16_bits(rng.normal(0, 3, (n, V)))
    out, ref, rows = run_both(traj, turn, mask, zs, zt, grad_rows=list(range(0, n, 97)))
    check_all(out, ref, mask, 1.0, rows)
    # 1-token segments: every token its own (trajectory, turn)
    n = 2500
    traj = (np.arange(n) // 50).astype(np.int32)
    turn = (np.arange(n) % 50).astype(np.int32)
    mask = (rng.uniform(size=n) < 0.5).astype(np.uint8)
    zs = bf16_bits(rng.normal(0, 3, (n, V)))
    zt = bf16_bits(rng.normal(0, 3, (n, V)))
    out, ref, rows = run_both(traj, turn, mask, zs, zt, max_turns=50,
                              grad_rows=list(range(0, n, 89)))
    check_all(out, ref, mask, 1.0, rows)


def test_trajectory_with_thousands_of_turns(gpu):
    """One trajectory of 2,600 one-token turns, then one of 400: the segments
    of the first lie up to 2,599 segments after their trajectory's first, so
    the search for each segment's head leaves the 2,048 segment ids a
    workgroup holds in LDS."""
    rng = np.random.default_rng(48)
    V, n1, n2 = 64, 2600, 400
    traj = np.concatenate([np.zeros(n1, np.int32), np.ones(n2, np.int32)])
    turn = np.concatenate([np.arange(n1), np.arange(n2)]).astype(np.int32)
    mask = (rng.uniform(size=n1 + n2) < 0.7).astype(np.uint8)
    zs = bf16_bits(rng.normal(0, 3, (n1 + n2, V)))
    zt = bf16_bits(rng.normal(0, 3, (n1 + n2, V)))
    out, ref, rows = run_both(traj, turn, mask, zs, zt, max_turns=n1,
                              grad_rows=list(range(0, n1 + n2, 37)))
    check_all(out, ref, mask, 1.0, rows)


def test_batch_beyond_the_fused_scan(gpu):
    """2,200,000 tokens: more than 2,048 tiles of 1,024 tokens, so the segment
    kernels take the separate scan of the tile counts instead of summing them
    in every workgroup.  Several thousand trajectories with padding between
    some turns, V = 16."""
    rng = np.random.default_rng(47)
    n_target, V = 2_200_000, 16
    lens = rng.integers(1, 120, size=n_target // 30)
    lens = lens[:np.searchsorted(np.cumsum(lens), n_target) + 1]
    turns_per_traj = rng.integers(1, 40, size=lens.size)
    traj_of_seg = np.repeat(np.arange(turns_per_traj.size), turns_per_traj)[:lens.size]
    turn_of_seg = np.concatenate([np.sort(rng.choice(60, size=k, replace=False))
                                  for k in turns_per_traj])[:lens.size]
    traj = np.repeat(traj_of_seg, lens).astype(np.int32)
    turn = np.repeat(turn_of_seg, lens).astype(np.int32)
    mask = (rng.uniform(size=traj.size) < 0.6).astype(np.uint8)
    # padding runs replace the first tokens of every 50th segment
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    for s0, ln in zip(starts[::50], lens[::50]):
        k = min(3, int(ln) - 1)
        traj[s0:s0 + k], turn[s0:s0 + k], mask[s0:s0 + k] = -1, 0, 0
    n = traj.size
    assert n > 2048 * 1024
    zs = bf16_bits(rng.normal(0, 3, (n, V)))
    zt = bf16_bits(rng.normal(0, 3, (n, V)))
    log(f"fallback scan: N={n} segments={lens.size}")
    out, ref, rows = run_both(traj, turn, mask, zs, zt, max_turns=60,
                              grad_rows=list(range(0, n, 4099)))
    assert ref.status == O.OK
    check_all(out, ref, mask, 1.0, rows)


def test_extreme_but_finite_logits(gpu):
    traj, turn, mask, zs, zt = make_batch(43, V=2048, dtype="f32", sigma=20.0, noise=5.0)
    zs[::3] -= 1e4
    zt[1::3] += 80.0
    out, ref, rows = run_both(traj, turn, mask, zs, zt)
    check_all(out, ref, mask, 1.0, rows)


def _as(dtype, x):
    return bf16_bits(x) if dtype == "bf16" else np.asarray(x, np.float32)


@pytest.mark.parametrize("dtype,vpt", [("f32", 0), ("bf16", 0), ("bf16", 2)])
def test_spike_beyond_the_sampled_reference(dtype, vpt, gpu):
    """One logit far above every thread's first pack overflows the fast
    path's sums (2^(150 log2 e) > FLT_MAX); the chunk is redone against its
    exact maximum."""
    traj, turn, mask, zs, zt = make_batch(44, V=32000, dtype="f32")
    rng = np.random.default_rng(7)
    n = zs.shape[0]
    cols = rng.integers(4096, 32000, n)
    r = np.arange(n)
    zs[r[0::3], cols[0::3]] += 150.0
    zt[r[1::3], cols[1::3]] += 150.0
    zs[r[2::3], cols[2::3]] += 150.0
    zt[r[2::3], cols[2::3]] += 149.0
    out, ref, rows = run_both(traj, turn, mask, _as(dtype, zs), _as(dtype, zt), vpt=vpt)
    check_all(out, ref, mask, 1.0, rows)


@pytest.mark.parametrize("dtype,vpt", [("bf16", 2), ("f32", 1), ("bf16", 0)])
def test_rows_mixing_fast_and_offset_chunks(dtype, vpt, gpu):
    """Row offsets of 50..69: some chunks of a row see a sampled maximum above
    64 and take the offset path, their row mates do not; the merge and the
    gradient must treat both forms alike."""
    traj, turn, mask, zs, zt = make_batch(45, V=32000, dtype="f32")
    off = (50.0 + np.arange(zs.shape[0]) % 20)[:, None].astype(np.float32)
    out, ref, rows = run_both(traj, turn, mask, _as(dtype, zs + off), _as(dtype, zt + off + 0.5),
                              vpt=vpt)
    check_all(out, ref, mask, 1.0, rows)


@pytest.mark.parametrize("shift_s,shift_t,dtype", [(5000.0, 5000.0, "f32"), (-3000.0, 3000.0, "f32"),
                                                   (1000.0, 1000.0, "bf16"), (-96.0, 0.0, "bf16"),
                                                   (1e6, -1e6, "f32"), (1e30, -1e30, "f32")])
def test_large_logit_offsets_keep_full_accuracy(shift_s, shift_t, dtype, gpu):
    """KL and its gradient do not depend on a constant added to a row of
    either model; computed against the chunk references they keep the same
    accuracy however large the offsets are."""
    traj, turn, mask, zs, zt = make_batch(46, V=4096, dtype="f32")
    out, ref, rows = run_both(traj, turn, mask, _as(dtype, zs + shift_s), _as(dtype, zt + shift_t))
    check_all(out, ref, mask, 1.0, rows)


# ----------------------------------------------------------------------------
# data errors detected on the device


def test_concurrent_calls_on_two_streams(gpu):
    """Two calls with distinct workspaces, enqueued on two streams at once,
    give bit for bit what the same calls give one after the other (the row
    kernels' exchanges and tickets are per workspace)."""
    log("two concurrent calls")
    batches = []
    for seed in (70, 71):
        traj, turn, mask, zs_h, zt_h = make_batch(seed, n_traj=60, max_turns=6, V=32000,
                                                  dtype="bf16", max_len=30)
        zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
        ids = ids_to_device(traj, turn, mask)
        batches.append((zs, zt) + ids + (len(traj),))

    def run(b, grad, stats, kl, ws):
        zs, zt, turn_d, traj_d, mask_d, n = b
        loss, _, _, _, _ = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.4, grad=grad, max_turns=8,
                                     turn_stats=stats, token_kl=kl, workspace=ws, check=False)
        return loss

    T.set_row_tiling(3)  # six chunks per row
    try:
        outs = []
        for mode in ("sequential", "concurrent"):
            bufs = [(torch.empty_like(b[0]), T.new_turn_stats(8),
                     torch.empty(b[5], dtype=torch.float32, device="cuda"),
                     T.Workspace(b[5], 32000, T.BF16, 8)) for b in batches]
            torch.cuda.synchronize()
            if mode == "sequential":
                losses = [run(b, *bf) for b, bf in zip(batches, bufs)]
            else:
                streams = [torch.cuda.Stream(), torch.cuda.Stream()]
                losses = []
                for st, b, bf in zip(streams, batches, bufs):
                    st.wait_stream(torch.cuda.current_stream())
                    with torch.cuda.stream(st):
                        losses.append(run(b, *bf))
                for st in streams:
                    torch.cuda.current_stream().wait_stream(st)
            torch.cuda.synchronize()
            for bf in bufs:
                assert bf[3].status() == T.OK
            outs.append([(l.cpu(), bf[0].view(torch.int16).cpu(), bf[1].cpu(), bf[2].cpu())
                         for l, bf in zip(losses, bufs)])
    finally:
        T.set_row_tiling(0)
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            assert torch.equal(x, y)


def test_exchange_timeout_is_reported_and_the_workspace_recovers(gpu):
    """A bound of one poll on the row kernel's wait for its row mates (set
    from the host) makes multi-chunk rows time out: the call reports
    TURNKL_ERR_SYNC_TIMEOUT, the loss is NaN, every kernel exits, and the next
    call on the same workspace, with the default bound, is correct."""
    log("exchange timeout forced from the host")
    traj, turn, mask, zs_h, zt_h = make_batch(90, n_traj=40, max_turns=6, V=32000,
                                              dtype="bf16", max_len=24)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    T.set_row_tiling(3)  # six chunks per row
    try:
        ws = T.Workspace(len(traj), 32000, T.BF16, 8)
        T.set_spin_limit(1)
        try:
            loss, _, _, _, _ = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.4, max_turns=8,
                                         workspace=ws, check=False)
            torch.cuda.synchronize()
        finally:
            T.set_spin_limit(0)
        assert ws.status() == T.ERR_SYNC_TIMEOUT
        assert torch.isnan(loss).all()
        stats = T.new_turn_stats(8)
        loss, g, _, kl, ws = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.4, max_turns=8,
                                       turn_stats=stats, token_kl=True, workspace=ws)
        torch.cuda.synchronize()
    finally:
        T.set_row_tiling(0)
    ref = O.fwd_bwd(traj, turn, mask, 0.4, 8, lambda r: (zs_h[r], zt_h[r]), O.DTYPE_BF16, 1.0,
                    list(range(0, len(traj), 7)))
    check_all((loss, g, stats, kl, ws), ref, mask, 1.0, list(range(0, len(traj), 7)))


@pytest.mark.parametrize("case", ["pad_mask", "turn_high", "turn_negative", "traj_down",
                                  "turn_down", "split_turn", "first_error_wins"])
def test_device_errors_match_oracle(case, gpu):
    traj, turn, mask, zs, zt = make_batch(50, pad=False, min_len=3)
    traj, turn, mask = traj.copy(), turn.copy(), mask.copy()
    n = len(traj)
    i = n // 2
    if case == "pad_mask":
        traj[i] = -1
        mask[i] = 1
    elif case == "turn_high":
        turn[i] = 8
    elif case == "turn_negative":
        turn[i] = -3
    elif case == "traj_down":
        traj[i:] = np.where(traj[i:] >= 0, traj[i:] - 100, traj[i:])
    elif case == "turn_down":  # a later turn of a trajectory with a smaller id
        seg = O.segments(traj, turn, mask, 8)
        s_ = next(k for k in range(1, seg.count)
                  if seg.traj[k] == seg.traj[k - 1] and seg.turn[k - 1] >= 1)
        lo, hi = seg.start[s_], seg.start[s_] + seg.length[s_]
        turn[lo:hi] = seg.turn[s_ - 1] - 1
    elif case == "split_turn":  # padding inside a turn makes two runs of one turn id
        seg = O.segments(traj, turn, mask, 8)
        s_ = next(k for k in range(seg.count) if seg.length[k] >= 3)
        j = seg.start[s_] + 1
        traj[j] = -1
        mask[j] = 0
    elif case == "first_error_wins":
        turn[i + 2] = 99
        traj[i] = -1
        mask[i] = 1
    ref = O.segments(traj, turn, mask, 8)
    assert ref.status != O.OK
    zs_d, zt_d = to_device_logits(zs), to_device_logits(zt)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    with pytest.raises(T.TurnKLError) as ei:
        T.fwd_bwd(zs_d, zt_d, turn_d, traj_d, mask_d, 0.5, max_turns=8)
    assert ei.value.code == ref.status, (case, ei.value.code, ref.status)
    loss, _, _, _, ws = T.fwd_bwd(zs_d, zt_d, turn_d, traj_d, mask_d, 0.5, max_turns=8,
                                  check=False)
    assert ws.status() == ref.status
    assert torch.isnan(loss).all()


def test_binding_rejects_undersized_or_mismatched_buffers(gpu):
    """The Python binding checks the size, dtype, shape and device of every
    caller buffer before calling the C ABI, which takes bare pointers."""
    traj, turn, mask, zs_h, zt_h = make_batch(97, n_traj=2, V=1024, dtype="bf16")
    n = len(traj)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    call = lambda **kw: T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, 0.5, max_turns=8, **kw)
    bad = [
        dict(turn_stats=T.new_turn_stats(7)),
        dict(success=torch.zeros(n, dtype=torch.uint8, device="cuda"),
             outcome_stats=T.new_turn_stats(15)),
        dict(token_kl=torch.empty(n - 1, dtype=torch.float32, device="cuda")),
        dict(token_kl=torch.empty(n, dtype=torch.float16, device="cuda")),
        dict(grad=torch.empty((n, 1000), dtype=torch.bfloat16, device="cuda")),
        dict(grad=torch.empty((n, 1024), dtype=torch.float32, device="cuda")),
        dict(token_lse=torch.empty((n, 2), dtype=torch.float32)),
        dict(token_weights=torch.empty(n - 1, dtype=torch.float32, device="cuda")),
    ]
    for kw in bad:
        with pytest.raises((ValueError, TypeError)):
            call(**kw)
    with pytest.raises(ValueError):
        T.fwd_bwd(zs, zt[:-1], turn_d, traj_d, mask_d, 0.5, max_turns=8)
    ids = torch.zeros((n, 4), dtype=torch.int32, device="cuda")
    vals = torch.zeros((n, 4), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):
        T.fwd_bwd_topk(zs, ids, vals, turn_d, traj_d, mask_d, 0.5, max_turns=8,
                       grad_topk=torch.empty((n, 3), dtype=torch.float32, device="cuda"))
    # the same call with correct buffers still works
    loss, *_ = call(turn_stats=T.new_turn_stats(8), token_kl=True)
    torch.cuda.synchronize()
    assert torch.isfinite(loss).all()
