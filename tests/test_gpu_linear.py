"""The single-linear entry point of the co-run study (nova_linear) against the oracle's linear:
every kernel variant the study co-runs, out += x w^T with bf16 inputs and fp32 accumulation,
including ragged row counts; and the shape checks that refuse what a variant does not cover."""
import numpy as np
import pytest

from oracle import vlm
from paper_2509_21301_amd import synth

pytestmark = pytest.mark.gpu

TOL = 1e-4     # fp32 accumulation of exact bf16 products, compared norm-wise with float64


def _case(m, k, n, seed):
    x = synth.normal((m, k), seed, f"lin_x{m}x{k}", std=1.0)
    w = synth.normal((n, k), seed, f"lin_w{n}x{k}", std=0.05)
    return x, w


@pytest.mark.parametrize("variant,m,k,n", [(0, 300, 1280, 512), (0, 1500, 1024, 2304), (1, 300, 1280, 512),
                                           (2, 3, 1024, 16384), (2, 20, 512, 16384), (3, 3, 1024, 1000),
                                           (3, 1, 3584, 512), (3, 4, 512, 96)])
def test_linear_variants_match_oracle(gpu_lib, variant, m, k, n):
    import torch
    nova = gpu_lib
    x, w = _case(m, k, n, seed=variant + 1)
    xd = torch.from_numpy(x).cuda().to(torch.bfloat16)
    wd = torch.from_numpy(w).cuda().to(torch.bfloat16)
    base = synth.normal((m, n), 9, f"lin_o{m}x{n}", std=1.0)
    out = torch.from_numpy(base).cuda()
    nova.linear(variant, xd, wd, out)
    torch.cuda.synchronize()
    ref = base + vlm.linear(x, w)
    assert vlm.max_rel_err(out.cpu().numpy(), ref) < TOL


def test_linear_shape_checks(gpu_lib):
    import torch
    nova = gpu_lib
    x = torch.zeros(5, 512, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(2048, 512, dtype=torch.bfloat16, device="cuda")
    out = torch.zeros(5, 2048, dtype=torch.float32, device="cuda")
    with pytest.raises(nova.NovaError) as e:
        nova.linear(nova.LINEAR_THIN_VALU, x, w, out)          # more than 4 rows
    assert e.value.code == nova.EUNSUPPORTED
    with pytest.raises(nova.NovaError) as e:
        nova.linear(nova.LINEAR_THIN, x, w, out)               # 32 row groups would split K on 256 CUs
    assert e.value.code == nova.EUNSUPPORTED
    with pytest.raises(nova.NovaError):
        nova.linear(7, x, w, out)
