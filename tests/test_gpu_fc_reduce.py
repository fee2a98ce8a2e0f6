"""GPU parity of hdf_fc_reduce (the generic dense fc reducer, Sec. 2.2 / Table 1)
against the oracle: bf16 outputs within the bf16 storage tolerance, fp32 within 1e-4
relative per row."""
import numpy as np
import pytest
import torch

import synth
from oracle.fc_reducer import fc_reduce as ref_fc
from oracle.numerics import as_f64
from paper_2606_26744_amd import hdf
from tests._tol import assert_bf16_close, assert_f32_rows_close

pytestmark = pytest.mark.gpu


def _case(n, m, d, dtype, seed, bias=True):
    print(f"[fc_reduce] n={n} m={m} d={d} dtype={dtype} bias={bias}", flush=True)
    H = synth.normal([n, m, d], 1.0, seed, 70, dtype=dtype, device="cuda")
    W = synth.normal([d, m * d], 0.02, seed, 71, dtype=dtype, device="cuda")
    b = synth.normal([d], 0.1, seed, 72, dtype="f32", device="cuda") if bias else None
    Y = hdf.fc_reduce(H, hdf.pack_weight(W), b)
    torch.cuda.synchronize()
    ref = ref_fc(synth.to_numpy_bits(H), synth.to_numpy_bits(W),
                 None if b is None else b.cpu().numpy(), dtype=dtype)
    got = synth.to_numpy_bits(Y)
    if dtype == "bf16":
        assert_bf16_close(as_f64(got), ref, "Y")
    else:
        assert_f32_rows_close(got, ref, "Y")


def test_warm_step_rows():
    """The full-size step's 128 new rows: 4 paths x 4096 (a 67M-parameter projection)."""
    _case(128, 4, 4096, "bf16", 1)


@pytest.mark.parametrize("n,m,d,dtype,bias", [(37, 4, 256, "f32", True), (300, 3, 1024, "bf16", False),
                                              (1, 8, 512, "bf16", True), (2050, 2, 128, "bf16", True),
                                              # more than 128 rows on the matrix-core tiles with
                                              # K = 64 and 128: fewer 32-wide K units than the
                                              # weight ring holds, and exactly as many
                                              (257, 1, 64, "bf16", False), (300, 2, 64, "bf16", True)])
def test_shapes(n, m, d, dtype, bias):
    _case(n, m, d, dtype, n + m, bias)


def test_rows_past_one_chunk():
    """More rows than one projection launch takes (16384): the chunks line up."""
    _case(16384 + 100, 2, 256, "bf16", 3)


def test_block_identity_weights_sum_the_paths():
    """W_fc = [I I I I] sums the paths exactly as the gated reducer with unit gates."""
    n, m, d = 64, 4, 512
    H = synth.normal([n, m, d], 1.0, 9, 70, dtype="f32", device="cuda")
    W = torch.cat([torch.eye(d, device="cuda")] * m, dim=1).contiguous()
    Y = hdf.fc_reduce(H, hdf.pack_weight(W))
    torch.cuda.synchronize()
    assert torch.allclose(Y, H.sum(dim=1), rtol=1e-6, atol=1e-5)


def test_empty():
    H = torch.empty((0, 4, 256), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((256, 1024), dtype=torch.bfloat16, device="cuda")
    assert hdf.fc_reduce(H, hdf.pack_weight(W)).shape == (0, 256)
