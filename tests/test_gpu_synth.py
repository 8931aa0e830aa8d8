"""The device generator writes the same bits as the host generator, so inputs
generated in HBM are the inputs the CPU oracle regenerates on the host."""
import numpy as np
import pytest
import torch

import synth
from gpu_support import log, rows_bits_to_host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_device_generator_matches_host_bits(name, gpu):
    w = synth.make(name)
    log(f"synth {name}: N={w.n_tokens} V={w.vocab}")
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([[0, w.n_tokens - 1],
                                     rng.integers(0, w.n_tokens, size=6)])).astype(np.int64)
    # generate only the sampled rows on the device, with a padded row stride
    ld = w.vocab + 24
    dt = torch.bfloat16 if w.dtype == synth.configs.BF16 else torch.float32
    zs = torch.empty((len(rows), ld), dtype=dt, device=gpu)
    zt = torch.empty((len(rows), ld), dtype=dt, device=gpu)
    ts = torch.from_numpy(w.teacher_sigma).to(gpu)
    stream = torch.cuda.current_stream().cuda_stream
    es = 2 if dt == torch.bfloat16 else 4
    for k, r in enumerate(rows.tolist()):
        synth._lib.fill_device(w.params(ld), ts.data_ptr(), r, r + 1,
                               zs.data_ptr() + k * ld * es, zt.data_ptr() + k * ld * es, stream)
    torch.cuda.synchronize()
    hs, ht = w.host_rows(rows)
    ds = rows_bits_to_host(zs[:, :w.vocab], np.arange(len(rows)))
    dtt = rows_bits_to_host(zt[:, :w.vocab], np.arange(len(rows)))
    assert np.array_equal(ds, hs) and np.array_equal(dtt, ht)
