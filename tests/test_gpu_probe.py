"""The MFMA-rate measurement aid (cw_probe_mfma_bf16) does the work it declares:
with all-one fragments every accumulator element gains 16 per instruction, so
each thread's sum after `iters` rounds of 8 instructions is exactly
8 x 16 x 16 x iters; with random fragments the sums are finite."""
import pytest
import torch

from paper_2606_19667_amd import cw, inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("iters,workgroups", [(1, 1), (7, 3), (64, 300)])
def test_probe_ones_exact(iters, workgroups):
    print(f"probe ones iters={iters} workgroups={workgroups}", flush=True)
    ops = torch.ones(6 * 512 + 512 * 5, dtype=torch.bfloat16, device="cuda")
    sink = torch.full((workgroups * 512,), -1.0, dtype=torch.float32, device="cuda")
    cw.probe_mfma_bf16(ops, sink, iters, workgroups)
    torch.cuda.synchronize()
    assert torch.all(sink == float(8 * 16 * 16 * iters))


def test_probe_random_finite():
    print("probe random", flush=True)
    ops = inputs.normal_bf16((0, 301), (4096 * 512,), "cuda")
    sink = torch.empty(16 * 512, dtype=torch.float32, device="cuda")
    cw.probe_mfma_bf16(ops, sink, 50, 16)
    torch.cuda.synchronize()
    assert torch.isfinite(sink).all()
    assert sink.abs().max().item() > 0
