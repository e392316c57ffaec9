"""FP8 (e4m3) quantiser and linear layer on the GPU against oracle.fp8:
codes and scales bit-exact (an integer decision taken in fp32 on both
sides), the linear layer's output within its own fp32 accumulation and
storage rounding of the exact product of the same codes (Section 3.5.2)."""
import numpy as np
import pytest
import torch

import synth
from oracle import fp8 as ofp8
from oracle.metrics import max_rel_err
from tests._util import DEV, to_dev

QCASES = {
    # name: (rows, cols, dtype, rowwise)
    "rows-bf16-2208": (300, 2208, "bf16", True),
    "rows-f32-ragged": (257, 77, "f32", True),
    "tensor-bf16-1024": (129, 1024, "bf16", False),
    "tensor-f32-odd": (7, 13, "f32", False),
    "rows-bf16-one-col": (64, 1, "bf16", True),
}


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(QCASES))
def test_fp8_quantize_bit_exact(name):
    from paper_2512_09200_amd import api
    rows, cols, dt, rowwise = QCASES[name]
    print(f"[fp8-quant] {name}", flush=True)
    r = np.random.default_rng(5)
    x = (r.standard_normal((rows, cols)) * np.exp2(r.integers(-10, 10, (rows, 1)))).astype(np.float32)
    x[1] = 0.0
    x[2, 0] = -0.0
    x = synth.to_storage(x, dt).float().numpy()
    q, s = api.lattice_fp8_quantize(to_dev(x, synth.torch_dtype(dt)), "row" if rowwise else "tensor")
    torch.cuda.synchronize()
    qr, sr = ofp8.quantize(x, rowwise)
    np.testing.assert_array_equal(s.cpu().numpy(), sr)
    qg = q.cpu().numpy()
    np.testing.assert_array_equal(qg[:, :cols], qr)
    assert not np.any(qg[:, cols:])                      # row padding written as zeros


LCASES = {
    # name: (M, N, K, relu, out dtype, a rowwise, w rowwise)
    "top-layer1-shape": (1024, 1024, 2208, True, "bf16", True, True),
    "ragged": (300, 200, 77, True, "bf16", True, True),
    "tensorwise-fp32-out": (257, 136, 512, False, "f32", False, False),
    "mixed-scales": (130, 260, 1040, True, "bf16", True, False),
    "k-one-step": (64, 64, 16, False, "f32", True, True),
}


@pytest.mark.gpu
@pytest.mark.parametrize("fast", [False, True], ids=["precise", "fast"])
@pytest.mark.parametrize("name", list(LCASES))
def test_fp8_linear(name, fast):
    """Codes bit-exact; the output within oracle.fp8.linear_fp8_bound (the
    matrix instruction's measured alignment, fp32 adds and scale products)
    of the exact product of the same codes, plus the output's own rounding."""
    from paper_2512_09200_amd import api
    M, N, K, relu, odt, arow, wrow = LCASES[name]
    print(f"[fp8-linear] {name} fast_accum={fast}", flush=True)
    r = np.random.default_rng(6)
    x = synth.to_storage(r.standard_normal((M, K)).astype(np.float32), "bf16").float().numpy()
    w = synth.to_storage((r.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32), "bf16").float().numpy()
    b = (r.standard_normal(N) * 0.1).astype(np.float32)
    qa, sa = api.lattice_fp8_quantize(to_dev(x, torch.bfloat16), "row" if arow else "tensor")
    qw, sw = api.lattice_fp8_quantize(to_dev(w, torch.bfloat16), "row" if wrow else "tensor")
    y = api.lattice_linear_fp8_fwd(qa, sa, qw, sw, K, bias=to_dev(b), relu=relu, fast_accum=fast,
                                   out_dtype=torch.bfloat16 if odt == "bf16" else torch.float32)
    torch.cuda.synchronize()
    qar, sar = ofp8.quantize(x, arow)
    qwr, swr = ofp8.quantize(w, wrow)
    np.testing.assert_array_equal(qa.cpu().numpy()[:, :K], qar)
    np.testing.assert_array_equal(qw.cpu().numpy()[:, :K], qwr)
    ref = ofp8.linear_fp8(qar, sar, qwr, swr, b, relu=relu)     # ReLU is 1-Lipschitz
    bound = ofp8.linear_fp8_bound(qar, sar, qwr, swr, b, fast_accum=fast)
    us = 2.0 ** -8 if odt == "bf16" else 0.0
    bound = bound + us * (np.abs(ref) + bound) + 1e-37
    got = y.float().cpu().double().numpy()
    diff = np.abs(got - ref)
    rms = np.sqrt(np.mean(diff ** 2) / np.mean(ref ** 2))
    print(f"  worst |x-r|/bound={np.max(diff / bound):.3f}, rms error/rms={rms:.2e}, "
          f"max_rel_err={max_rel_err(got, ref):.2e}", flush=True)
    assert np.all(np.isfinite(got))
    assert np.all(diff <= bound)
    if not fast:
        assert max_rel_err(got, ref) <= 2e-2
